// Split-KV decode sweep over a paged grouped-query KV cache (gfx950).
//
// Computes, for every (request b, shard s, query head h), the pair (O, ln Z) of the shard's cached
// positions (Q-First, arXiv:2608.15473, §5: Z = sum exp(s_i), O = sum exp(s_i) v_i / Z, scores
// s_i = scale * q . k_i as in §2).  The kernel is bound by HBM bandwidth: every cached byte of K
// and V is read exactly once, and the G query heads that share a KV head are all served from that
// one read.
//
// Work decomposition.  One workgroup = one unit (b, s, c, g): KV head g of chunk c of shard s of
// request b (chunks > 1 only when a shape has too few units to fill the GPU).  Its W wavefronts
// take the unit's pages round-robin.  Inside a wavefront the 64 lanes form 4 rows of 16; a page
// (16 positions x 128 dims of bf16 = 4 KB per tensor) is read with 4 fully coalesced 16-byte
// loads per lane, load j covering positions 4j..4j+3, so lane (row r, column c) holds dims
// 8c..8c+7 of position 4j + r.  Each row is an independent online-softmax sweeper over the
// positions r, r+4, r+8, r+12 of every page; rows and wavefronts merge once, at the end.
//
// Per page and lane, scores: at G = 4 or 8 query heads per KV head, on the matrix cores (the K
// tile passes through LDS into the operand layout of four v_mfma_f32_16x16x32_bf16, which leave
// each lane the scores of exactly the positions whose V it holds, for one head; the other heads'
// come from neighbouring lanes by DPP); otherwise with v_dot2c_f32_bf16 on the packed bf16 pairs and a 16-lane
// DPP all-reduce per score.  Both take exact bf16 products and fp32 sums.  Then exp2 in the log2
// domain and fp32 FMAs for PV with the bf16 values unpacked by shift/mask.  The running max is
// raised lazily (only when a score exceeds it by more than kLazy), so the O rescale is rare after
// a shard's first pages.
#include <math.h>

#include <atomic>

#include "linear_body.h"
#include "merge_body.h"
#include "qf_internal.h"

namespace qf {
namespace {

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

constexpr int D = kHeadDim;
constexpr int P = kPage;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kNonTemporal = 2;  // buffer-load cache-policy bit "nt" on gfx950
constexpr float kLazy = 8.0f;  // log2 units: p = exp2(s - m) stays <= 256 between rescales

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

using mrg::row_sum16;  // sum over the 16 lanes of a DPP row, the same bits on each

// Lane 4*(c/4) + h's value in every lane c of its quad (DPP quad_perm [h,h,h,h]).
__device__ __forceinline__ float quad_bcast(float x, int h) {
  const int v = __float_as_int(x);
  switch (h) {
    case 0: return __int_as_float(__builtin_amdgcn_mov_dpp(v, 0x00, 0xF, 0xF, true));
    case 1: return __int_as_float(__builtin_amdgcn_mov_dpp(v, 0x55, 0xF, 0xF, true));
    case 2: return __int_as_float(__builtin_amdgcn_mov_dpp(v, 0xAA, 0xF, 0xF, true));
    default: return __int_as_float(__builtin_amdgcn_mov_dpp(v, 0xFF, 0xF, 0xF, true));
  }
}

// Lane 8*(c/8) + h's value in every lane c of its 8-lane group (G = 8), or the quad's (G <= 4),
// for the matrix path, where lane c holds the values of head c % G.  For G = 8 the quad broadcast
// gives one half of each 8-lane group the right head, and a 4-lane row shift written only into
// the other half's DPP banks (quads) completes it.
template <int G>
__device__ __forceinline__ float group_bcast(float x, int h) {
  if constexpr (G == 1) {
    return x;
  } else if constexpr (G <= 4) {
    return quad_bcast(x, h);
  } else {
    const float t = quad_bcast(x, h & 3);
    return h < 4 ? __builtin_amdgcn_update_dpp(t, t, 0x114, 0xF, 0xA, false)   // row_shr:4 -> quads 1, 3
                 : __builtin_amdgcn_update_dpp(t, t, 0x104, 0xF, 0x5, false);  // row_shl:4 -> quads 0, 2
  }
}

// 16-byte slot of chunk `ch` (dims 8ch..8ch+7) of position `pos` in a wavefront's 4 KB K tile in
// LDS.  The XOR swizzle makes both the row-wise writes and the column-wise operand reads free of
// bank conflicts: a position's 16 chunks stay in its 256 bytes, and the 16 positions read together
// for one chunk land in 16 different slots of their rows.
__device__ __forceinline__ int kslot(int pos, int ch) {
  return pos * 16 + (ch ^ (4 * (pos & 3) + (pos >> 2)));
}

// Block-table entries are wave-uniform: read them through the constant address space so they
// become scalar loads (own counter), never vector loads that would join the page loads' vmcnt.
typedef const __attribute__((address_space(4))) int32_t* const_i32_ptr;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ void unpack8(const uint4& w, float* f) {
  f[0] = bf16_lo(w.x); f[1] = bf16_hi(w.x);
  f[2] = bf16_lo(w.y); f[3] = bf16_hi(w.y);
  f[4] = bf16_lo(w.z); f[5] = bf16_hi(w.z);
  f[6] = bf16_lo(w.w); f[7] = bf16_hi(w.w);
}

// Sweep and merge in one launch: every unit of a (request, KV head) counts itself in once its
// partial states are stored; the unit that completes the count merges the group's G query heads
// over all max_shards x chunks slots with the merge kernels' own code (merge_body.h).  The XCDs'
// L2 caches are not coherent with each other, and a device-scope fence would write back and
// invalidate a whole L2 per workgroup, so no fence is used: the partial states are written and
// read with device-scope accesses (which go through to the coherent level), every wavefront waits
// until its own stores have completed before the workgroup barrier, and the count is a
// device-scope atomic.  The last unit then sets the counter back to 0 for the next call.
// Nothing ever waits for another workgroup.
// The G query heads of one (request, KV head) merged over their `entries` slots by the last unit
// of the group.  When one 16-slot group per wavefront covers the slots with W / G wavefronts per
// head (or W / 2, ...), heads are merged side by side by teams of wavefronts, and every wavefront
// loads its log-partitions and O rows at once (one memory round trip; the O rows of empty slots
// are read and discarded); each team sums exactly what merge_row's wavefronts sum, with the same
// code (mrg::WaveMerge), so the bits are merge_row's.  Otherwise head by head with merge_row.  The partial states
// were written by other workgroups of this launch: read with device-scope loads.
template <int G, int W>
__device__ __forceinline__ void merge_group(const float* __restrict__ part_o,
                                            const float* __restrict__ part_lse,
                                            uint16_t* __restrict__ merged_o,
                                            float* __restrict__ merged_lse, int b, int g, int hq,
                                            int entries) {
  constexpr int K = mrg::K;
  const int groups = (entries + K - 1) / K;
  const int hpw = min(G, W / max(groups, 1));   // heads merged side by side
  if (hpw < 2) {
#pragma unroll 1
    for (int h = 0; h < G; ++h)
      mrg::merge_row<true, false, W, true>(part_o, part_lse, merged_o, merged_lse, entries, hq, b,
                                           g * G + h, nullptr, nullptr, nullptr, 1, 0.0f);
    return;
  }
  const int wph = W / hpw;                       // wavefronts per head, >= groups
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int sub = wave / wph, wl = wave % wph;
  const bool in_team = sub < hpw;
  const int i0 = K * wl;
  __shared__ mrg::WaveMergeLds<W> lds;
#pragma unroll 1
  for (int h0 = 0; h0 < G; h0 += hpw) {
    const int h = g * G + h0 + min(sub, hpw - 1);
    const float* lse = part_lse + (size_t)b * entries * hq + h;
    const float* o = part_o + ((size_t)b * entries * hq + h) * mrg::D + 2 * lane;
    const int32_t o_step = hq * mrg::D;
    const float* o_i0 = o + (size_t)i0 * o_step;
    float x = -INFINITY;
    if (in_team && lane < K && i0 + lane < entries)
      x = __hip_atomic_load(&lse[(size_t)(i0 + lane) * hq], __ATOMIC_RELAXED,
                            __HIP_MEMORY_SCOPE_AGENT);
    float2 v[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const bool in = in_team && i0 + k < entries;
      v[k] = __builtin_bit_cast(
          float2, in ? __hip_atomic_load(reinterpret_cast<const uint64_t*>(o_i0 + k * o_step),
                                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                     : 0ull);
    }
    // This wavefront's group, as one round of merge_row's loop.
    mrg::WaveMerge st;
    st.add(x, v);
    lds.put(wave, lane, st);
    __syncthreads();
    if (in_team && wl == 0) {   // the team's first wavefront: merge_row's final merge
      float lse_out;
      const float2 a = lds.finish(sub * wph, wph, lane, lse_out);
      const size_t out_idx = ((size_t)b * hq + h) * mrg::D / 2 + lane;
      reinterpret_cast<uint32_t*>(merged_o)[out_idx] = mrg::bf16_rne(a.x) | (mrg::bf16_rne(a.y) << 16);
      if (merged_lse && lane == 0) merged_lse[(size_t)b * hq + h] = lse_out;
    }
    __syncthreads();
  }
}

template <int G, int W>
__device__ __forceinline__ void merge_if_last(const float* __restrict__ part_o,
                                              const float* __restrict__ part_lse,
                                              int32_t* __restrict__ counters,
                                              uint16_t* __restrict__ merged_o,
                                              float* __restrict__ merged_lse, int b, int g,
                                              int hq, int hkv, int entries) {
  __shared__ int s_last;
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wavefront's partial stores are complete
  __syncthreads();
  if (threadIdx.x == 0) {
    const int prev = __hip_atomic_fetch_add(&counters[(size_t)b * hkv + g], 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    s_last = (prev == entries - 1);
  }
  __syncthreads();
  if (!s_last) return;
  merge_group<G, W>(part_o, part_lse, merged_o, merged_lse, b, g, hq, entries);
  if (threadIdx.x == 0)
    __hip_atomic_store(&counters[(size_t)b * hkv + g], 0, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

// Pages [p0, p1) of shard s of request b (the split rule of the interface: K = ceil(pages / S_b)
// whole pages per shard, the last ones shorter or empty), with the request's shape checked: an out-of-range
// context length or shard count is clamped (so nothing is read out of bounds) and reported in
// `poison`.  n is the clamped context length.
struct ShardRange {
  int n, p0, p1;
  bool poison;
};
__device__ __forceinline__ ShardRange shard_range(const int32_t* __restrict__ ctx_lens,
                                                 const int32_t* __restrict__ n_shards, int b,
                                                 int s, int32_t max_pages, int32_t max_shards) {
  ShardRange r;
  int n = ctx_lens[b];
  int S = n_shards[b];
  r.poison = false;
  const int cap = max_pages * P;
  if (n < 0 || n > cap) { r.poison = true; n = n < 0 ? 0 : cap; }
  if (S < 1 || S > max_shards) { r.poison = true; S = S < 1 ? 1 : max_shards; }
  const int pages = (n + P - 1) / P;
  const int per = (pages + S - 1) / S;
  r.n = n;
  r.p0 = r.p1 = 0;
  if (s < S) {
    r.p0 = (int)min((int64_t)s * per, (int64_t)pages);
    r.p1 = (int)min((int64_t)(s + 1) * per, (int64_t)pages);
  }
  return r;
}

// The sweep of one unit by one workgroup; `bid` plays the role of the workgroup index (it is the
// index itself in decode_split_kernel, the sweep's share of the indices in a shared launch).
// With MERGE, the unit also takes part in the fused merge (merge_if_last).
template <int G, int W, int NBUF, bool MERGE = false>
__device__ __forceinline__ void sweep_unit(
    const uint16_t* __restrict__ qp, const uint16_t* __restrict__ kp,
    const uint16_t* __restrict__ vp, const int32_t* __restrict__ block_table,
    const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ n_shards,
    float* __restrict__ out_o, float* __restrict__ out_lse, int32_t hq, int32_t hkv,
    int32_t max_pages, int32_t num_pages, int32_t max_shards, int32_t chunks, int32_t n_units,
    int32_t units_per_xcd, int32_t batch, int32_t order, float scale_log2, const unsigned bid,
    int32_t* __restrict__ counters = nullptr, uint16_t* __restrict__ merged_o = nullptr,
    float* __restrict__ merged_lse = nullptr, const int32_t* __restrict__ unit_order = nullptr) {
  // Which unit this workgroup sweeps.  Workgroups are dispatched in index order, round-robin over
  // the 8 XCDs.
  //  * Short shards (kOrderByRequest): each XCD takes a contiguous range of units in (request,
  //    shard, chunk, KV head) order, so a request's query, context length and block-table lines
  //    stay in one XCD's L2 and the short workgroups' prologues hit there.
  //  * Long shards (kOrderByShardDesc): units in (shard descending, request, KV head) order,
  //    round-robin over the XCDs, so the largest shards (high indices exist only in long requests)
  //    start first and every XCD gets an even share; the small shards fill the tail.  With
  //    sub-shard chunks the chunk index runs fastest, so the chunks of a shard alternate between
  //    even- and odd-numbered XCDs (the unit index modulo 8 is the XCD), and their sizes are
  //    weighted by that parity (kXcdWeightEven / kXcdWeightOdd): measured on MI355X, odd-numbered
  //    XCDs stream 8-17% slower than even ones under the long-shard sweep, whatever KV head they
  //    read, so equal chunks leave the even XCDs idle while the odd ones finish.
  //    Without chunks (and with at most kRankMaxPairs (request, shard) pairs), a unit order
  //    written by rank_units_kernel replaces both: each workgroup index names its unit, longest
  //    shard first, and the odd XCDs get fewer of the long units.
  int g, c, s, b;
  int pair = 0;  // long shards with chunks: index of the (request, shard, KV head) in unit order
  if (order == kOrderByRequest) {
    const int unit = (int)(bid % 8u) * units_per_xcd + (int)(bid / 8u);
    if (unit >= n_units) return;
    g = unit % hkv;
    int rest = unit / hkv;
    c = rest % chunks;
    rest /= chunks;
    s = rest % max_shards;
    b = rest / max_shards;
  } else {
    const int unit = unit_order != nullptr ? unit_order[bid] : (int)bid;
    if (unit < 0 || unit >= n_units) return;
    int rest;
    if (chunks > 1) {
      c = unit % chunks;
      pair = unit / chunks;
      g = pair % hkv;
      rest = pair / hkv;
    } else {
      c = 0;
      g = unit % hkv;
      rest = unit / hkv;
    }
    b = rest % batch;
    s = max_shards - 1 - rest / batch;
  }

  // The request's shape, checked: an out-of-range value poisons this unit's log-sum-exp with NaN.
  const ShardRange range = shard_range(ctx_lens, n_shards, b, s, max_pages, max_shards);
  const int n = range.n;
  bool poison = range.poison;
  const int p0 = range.p0;
  const int len = range.p1 - p0;
  int c0, c1;
  if (order == kOrderByShardDesc && chunks > 1) {
    // Chunk j of this shard runs on an XCD of parity (pair * chunks + j) % 2; the pages before
    // chunk c weigh kXcdWeightEven per even-XCD chunk and kXcdWeightOdd per odd one.
    const int first_odd = (int)(((int64_t)pair * chunks) & 1);
    auto weight_before = [&](int cc) -> int64_t {
      const int64_t even = first_odd ? cc / 2 : (cc + 1) / 2;
      return even * kXcdWeightEven + (cc - even) * kXcdWeightOdd;
    };
    const int64_t total = weight_before(chunks);
    c0 = p0 + (int)((int64_t)len * weight_before(c) / total);
    c1 = p0 + (int)((int64_t)len * weight_before(c + 1) / total);
  } else {
    const int cper = (len + chunks - 1) / chunks;
    c0 = p0 + (int)min((int64_t)c * cper, (int64_t)len);
    c1 = p0 + (int)min((int64_t)(c + 1) * cper, (int64_t)len);
  }

  // An empty unit (a slot past the request's shards, or an empty shard or chunk) reads nothing:
  // its ln Z is -inf (NaN if the request's shape was out of range), its O is never read, so it
  // stops here, before the query loads and the merge.  (Ragged batches are mostly such units.)
  if (c0 >= c1) {
    if (threadIdx.x < G) {
      const size_t slot = (((size_t)b * max_shards + s) * chunks + c) * hq + (size_t)g * G;
      if constexpr (MERGE)
        __hip_atomic_store(&out_lse[slot + threadIdx.x], poison ? NAN : -INFINITY,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else
        __builtin_nontemporal_store(poison ? NAN : -INFINITY, &out_lse[slot + threadIdx.x]);
    }
    if constexpr (MERGE)
      merge_if_last<G, W>(out_o, out_lse, counters, merged_o, merged_lse, b, g, hq, hkv,
                          max_shards * chunks);
    return;
  }

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int row = lane >> 4;
  const int col = lane & 15;

  // With 4 or 8 heads per KV head the scores come from the matrix cores (process_mf below);
  // otherwise the VALU computes them (process_valu).  Measured: the matrix path is 1-5% faster at
  // G = 4 and 27-32% faster at G = 8, where the VALU path spends most of its issue slots on the
  // dot products and reductions, and 1-2.5% slower at G = 2, where the VALU has slack and the LDS
  // round trip only adds latency.
  constexpr bool MF = G >= 4;

  // Queries of the group.  VALU path: dims 8col..8col+7 of every head as packed bf16 pairs.
  // Matrix path: the queries are the 16 columns of the B operand of S^T = K Q^T (column c holds
  // head c % G), split over the dims in 4 steps of 32: lane (row, col) holds dims
  // 32kk + 8row .. 32kk + 8row + 7 of head col % G for step kk.
  uint32_t qv[G][4];
  bf16x8_t qb[4];
  if constexpr (MF) {
    const uint4* qrow = reinterpret_cast<const uint4*>(qp + ((size_t)b * hq + (size_t)g * G + col % G) * D);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) qb[kk] = __builtin_bit_cast(bf16x8_t, qrow[4 * kk + row]);
  } else {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const uint4 t = reinterpret_cast<const uint4*>(qp + ((size_t)b * hq + (size_t)g * G + h) * D)[col];
      qv[h][0] = t.x; qv[h][1] = t.y; qv[h][2] = t.z; qv[h][3] = t.w;
    }
  }

  // Online-softmax state.  VALU path: every lane keeps (m, l) of all G heads for its row.  Matrix
  // path: lane (row, col) keeps them for head col % G only (m1, l1); the other heads' values sit
  // in the same quad (8-lane group at G = 8) and are broadcast when needed.  acc: dims 8col..8col+7 of every head.
  float m[G], l[G], acc[G][8];
  float m1 = -INFINITY, l1 = 0.0f;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.0f;
  }

  const const_i32_ptr bt =
      block_table ? (const_i32_ptr)(block_table + (size_t)b * max_pages) : nullptr;
  const size_t page_stride = (size_t)hkv * P * D;  // elements between physical pages
  const uint16_t* kbase = kp + (size_t)g * P * D;
  const uint16_t* vbase = vp + (size_t)g * P * D;

  // This wavefront's pages: c0 + wave + i * W for i < mine.
  const int mine = (c1 - c0 > wave) ? (c1 - c0 - wave + W - 1) / W : 0;
  auto page_of = [&](int i) { return c0 + wave + i * W; };
  // Raw block-table entry of page i (read one page past the last one in flight; checked only when
  // used, so the scalar load's latency hides behind the pages in flight).
  auto entry = [&](int i) -> int {
    if (i >= mine) return 0;
    const int pg = page_of(i);
    return bt ? bt[pg] : b * max_pages + pg;
  };
  // One 4 KB page of one KV head through a buffer resource whose size covers the page's cached
  // positions only: loads past it return zeros, so a page that does not exist (size 0) costs no
  // traffic and keeps the prefetch below unconditional and the wait counts static, and the slots
  // past the last position of a partial page read as zeros instead of whatever the pool holds
  // there (a zero V meets a zero weight; the scores of those slots are set to -inf).  The loads
  // are non-temporal (cache policy nt): every cached byte is read exactly once per sweep, and on
  // gfx950 streaming reads marked nt reach a markedly higher share of HBM bandwidth than
  // default-policy reads.
  auto issue = [&](uint4* kk, uint4* vv, int ph, int i) {
    const bool live = i < mine;
    if ((unsigned)ph >= (unsigned)num_pages) {
      poison |= live;
      ph = 0;
    }
    const int bytes = live ? min(n - page_of(i) * P, P) * D * 2 : 0;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(kbase + (size_t)ph * page_stride), (short)0, bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(vbase + (size_t)ph * page_stride), (short)0, bytes, 0x00020000);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      kk[j] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rk, lane * 16, j * 1024, kNonTemporal));
#pragma unroll
    for (int j = 0; j < 4; ++j)
      vv[j] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rv, lane * 16, j * 1024, kNonTemporal));
  };

  // P V for the 4 positions of this row, weights pr[j][h] of position 4j + row.  (The slots past
  // the last position of a partial page were loaded as zeros and have zero weights.)
  auto accumulate = [&](uint4* vc, auto&& weight) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float vf[8];
      unpack8(vc[j], vf);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float p = weight(j, h);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(p, vf[e], acc[h][e]);
      }
    }
  };

  // Matrix path.  The page's K tile goes through this wavefront's 4 KB of LDS: the coalesced
  // loads give lane (row, col) dims 8col.. of position 4j + row, and the operand reads give lane
  // (row, col) dims 32kk + 8row.. of position pi(col) = 4(col % 4) + col / 4, so that the
  // 16 x 16 result S^T = K Q^T lands with lane (row, col) holding the scores of positions
  // 4i + row (i = 0..3), the very positions whose V this lane reads, for head col % G.  Four
  // v_mfma_f32_16x16x32_bf16 (exact bf16 products, fp32 sums) replace 4G dot products and 4G
  // 16-lane reductions per position quad.
  __shared__ uint4 s_k[MF ? W : 1][MF ? P * 16 : 1];
  auto process_mf = [&](uint4* kc, uint4* vc, int pg) {
    const int valid = n - pg * P;  // slots [0, valid) of this page are cached positions
    uint4* tile = s_k[wave];
#pragma unroll
    for (int j = 0; j < 4; ++j) tile[kslot(4 * j + row, col)] = kc[j];
    // LDS operations of one wavefront complete in order; the fence only keeps the compiler from
    // moving the operand reads above the writes of other lanes' slots.
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    const int pos = 4 * (col & 3) + (col >> 2);
    f32x4_t st = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          __builtin_bit_cast(bf16x8_t, tile[kslot(pos, 4 * kk + row)]), qb[kk], st, 0, 0, 0);
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");

    float sc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) sc[i] = st[i] * scale_log2;
    if (valid < P) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (4 * i + row >= valid) sc[i] = -INFINITY;
    }
    const float mx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
    const bool raise = mx > m1 + kLazy;
    float alpha = 1.0f;
    if (raise) {
      alpha = __builtin_amdgcn_exp2f(m1 - mx);  // m1 = -inf -> 0
      l1 *= alpha;
      m1 = mx;
    }
    if (__builtin_amdgcn_ballot_w64(raise)) {   // rare after a shard's first page
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float a = group_bcast<G>(alpha, h);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] *= a;
      }
    }
    const float base = (m1 == -INFINITY) ? 0.0f : m1;
    float pr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) pr[i] = __builtin_amdgcn_exp2f(sc[i] - base);
    l1 += (pr[0] + pr[1]) + (pr[2] + pr[3]);
    accumulate(vc, [&](int j, int h) { return group_bcast<G>(pr[j], h); });
  };

  auto process_valu = [&](uint4* kc, uint4* vc, int pg) {
    const int valid = n - pg * P;  // slots [0, valid) of this page are cached positions

    // Scores of this row's 4 positions for the G heads, log2 domain.
    float sc[4][G];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float d = dot2(kc[j].x, qv[h][0], 0.0f);
        d = dot2(kc[j].y, qv[h][1], d);
        d = dot2(kc[j].z, qv[h][2], d);
        d = dot2(kc[j].w, qv[h][3], d);
        sc[j][h] = row_sum16(d) * scale_log2;
      }
    }
    if (valid < P) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (4 * j + row >= valid) {
#pragma unroll
          for (int h = 0; h < G; ++h) sc[j][h] = -INFINITY;
        }
    }

    float pr[4][G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mx = fmaxf(fmaxf(sc[0][h], sc[1][h]), fmaxf(sc[2][h], sc[3][h]));
      if (mx > m[h] + kLazy) {
        const float alpha = __builtin_amdgcn_exp2f(m[h] - mx);  // m = -inf -> 0
        l[h] *= alpha;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] *= alpha;
        m[h] = mx;
      }
      const float base = (m[h] == -INFINITY) ? 0.0f : m[h];
#pragma unroll
      for (int j = 0; j < 4; ++j) pr[j][h] = __builtin_amdgcn_exp2f(sc[j][h] - base);
      l[h] += (pr[0][h] + pr[1][h]) + (pr[2][h] + pr[3][h]);
    }
    accumulate(vc, [&](int j, int h) { return pr[j][h]; });
  };

  // Rotation over NBUF register buffers: pages i+1 .. i+NBUF-1 stream in while page i is
  // computed.  Scalar loads may return out of order, so waiting for one waits for all: each
  // block-table entry is requested only after the previous one has been consumed by issue().
  uint4 kbuf[NBUF][4], vbuf[NBUF][4];
#pragma unroll
  for (int t = 0; t < NBUF - 1; ++t) issue(kbuf[t], vbuf[t], entry(t), t);
  // The query loads (issued first) must have landed before the loop, so that the only loads in
  // flight inside it are the page buffers; the first pages stay in flight meanwhile
  // (s_waitcnt vmcnt(8 * (NBUF - 1)), expcnt 7, lgkmcnt 15).
  constexpr int kAhead = 8 * (NBUF - 1);
  __builtin_amdgcn_s_waitcnt((kAhead & 0xF) | ((kAhead >> 4) << 14) | 0x0F70);
  int ph_next = entry(NBUF - 1);
  for (int i = 0; i < mine; i += NBUF) {
#pragma unroll
    for (int t = 0; t < NBUF; ++t) {
      const int ahead = i + t + NBUF - 1;
      issue(kbuf[(t + NBUF - 1) % NBUF], vbuf[(t + NBUF - 1) % NBUF], ph_next, ahead);
      ph_next = entry(ahead + 1);
      if (i + t >= mine) goto swept;
      if constexpr (MF)
        process_mf(kbuf[t], vbuf[t], page_of(i + t));
      else
        process_valu(kbuf[t], vbuf[t], page_of(i + t));
    }
  }
swept:
  if constexpr (MF) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      m[h] = group_bcast<G>(m1, h);
      l[h] = group_bcast<G>(l1, h);
    }
  }

  // Merge the 4 rows of the wavefront (lanes col, col+16, col+32, col+48 hold the same dims).
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float M = fmaxf(m[h], __shfl_xor(m[h], 16));
    M = fmaxf(M, __shfl_xor(M, 32));
    const float f = (M == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m[h] - M);
    float lh = l[h] * f;
    lh += __shfl_xor(lh, 16);
    lh += __shfl_xor(lh, 32);
    l[h] = lh;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float a = acc[h][e] * f;
      a += __shfl_xor(a, 16);
      a += __shfl_xor(a, 32);
      acc[h][e] = a;
    }
    m[h] = M;
  }

  // Merge the W wavefronts through LDS and write the unit's (O, ln Z).
  __shared__ float s_acc[W][G][D];
  __shared__ float s_m[W][G];
  __shared__ float s_l[W][G];
  __shared__ int s_bad[W];
  if (row == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) s_acc[wave][h][col * 8 + e] = acc[h][e];
  }
  // Any poisoned wavefront poisons the unit: a ballot per wavefront, met in LDS at the barrier
  // the merge needs anyway (cheaper in registers than __syncthreads_or, which rebuilds a flat
  // thread index from the y and z indices).
  const bool wave_bad = __builtin_amdgcn_ballot_w64(poison) != 0;
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) { s_m[wave][h] = m[h]; s_l[wave][h] = l[h]; }
    s_bad[wave] = wave_bad ? 1 : 0;
  }
  __syncthreads();
  int bad = 0;
#pragma unroll
  for (int w = 0; w < W; ++w) bad |= s_bad[w];

  const size_t slot = (((size_t)b * max_shards + s) * chunks + c) * hq + (size_t)g * G;
  for (int idx = threadIdx.x; idx < G * D; idx += 64 * W) {
    const int h = idx / D;
    const int d = idx % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < W; ++w) M = fmaxf(M, s_m[w][h]);
    float L = 0.0f, A = 0.0f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < W; ++w) {
        const float f = __builtin_amdgcn_exp2f(s_m[w][h] - M);
        L = fmaf(f, s_l[w][h], L);
        A = fmaf(f, s_acc[w][h][d], A);
      }
    } else {
      // No finite score: no position at all (every l is 0; an empty shard) or only NaN scores
      // (a NaN query element; l is NaN), which must come out NaN like any NaN input.
#pragma unroll
      for (int w = 0; w < W; ++w) L += s_l[w][h];
      A = L;
    }
    const bool nan_only = M == -INFINITY && __builtin_isnan(L);
    if (M != -INFINITY || nan_only) {
      // Non-temporal: a thin stream of default-policy writes interleaved with the sweep's
      // reads costs far more HBM time than its bytes (measured ~4% of the sweep).
      if constexpr (MERGE)   // read by another workgroup of this launch (merge_if_last)
        __hip_atomic_store(&out_o[(slot + h) * D + d], A / L, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      else
        __builtin_nontemporal_store(A / L, &out_o[(slot + h) * D + d]);
    }
    if (d == 0) {
      float lse = nan_only ? NAN : (M == -INFINITY) ? -INFINITY : (M + log2f(L)) * kLn2;
      if (bad) lse = NAN;
      if constexpr (MERGE)
        __hip_atomic_store(&out_lse[slot + h], lse, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else
        __builtin_nontemporal_store(lse, &out_lse[slot + h]);
    }
  }
  if constexpr (MERGE)
    merge_if_last<G, W>(out_o, out_lse, counters, merged_o, merged_lse, b, g, hq, hkv,
                        max_shards * chunks);
}

// Three wavefronts per SIMD with two page buffers (the long-shard sweep): the matrix path at G = 4
// needs the hint to stay within 168 registers (it does, without spills); deeper buffers take two.
template <int G, int W, int NBUF>
__global__ void __launch_bounds__(64 * W)
__attribute__((amdgpu_waves_per_eu(NBUF == 2 && G <= 4 ? 3 : 2)))
decode_split_kernel(const uint16_t* __restrict__ qp, const uint16_t* __restrict__ kp,
                    const uint16_t* __restrict__ vp, const int32_t* __restrict__ block_table,
                    const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ n_shards,
                    float* __restrict__ out_o, float* __restrict__ out_lse, int32_t hq,
                    int32_t hkv, int32_t max_pages, int32_t num_pages, int32_t max_shards,
                    int32_t chunks, int32_t n_units, int32_t units_per_xcd, int32_t batch,
                    int32_t order, float scale_log2, const int32_t* __restrict__ unit_order) {
  sweep_unit<G, W, NBUF>(qp, kp, vp, block_table, ctx_lens, n_shards, out_o, out_lse, hq, hkv,
                         max_pages, num_pages, max_shards, chunks, n_units, units_per_xcd, batch,
                         order, scale_log2, blockIdx.x, nullptr, nullptr, nullptr, unit_order);
}

// The XCD dealing cycle of rank_units_kernel: kXcdWeightEven : kXcdWeightOdd in lowest terms
// (27 : 23), one cycle holding that many entries of every even and every odd XCD, spread by
// smooth weighted round-robin so that every prefix of the cycle is near the weights.
constexpr int kXcdCycleMax = 256;
struct XcdCycle {
  int len;
  int count[8];                  // entries of XCD x in one cycle
  uint8_t xcd[kXcdCycleMax];     // XCD of entry i
  uint16_t before[kXcdCycleMax]; // entries of the same XCD before entry i
};
constexpr int gcd_of(int a, int b) { return b ? gcd_of(b, a % b) : a; }
constexpr XcdCycle make_xcd_cycle() {
  XcdCycle c{};
  const int gd = gcd_of(kXcdWeightEven, kXcdWeightOdd);
  const int we = kXcdWeightEven / gd, wo = kXcdWeightOdd / gd;
  c.len = 4 * (we + wo);
  int cur[8] = {};
  for (int i = 0; i < c.len; ++i) {
    int best = 0;
    for (int x = 0; x < 8; ++x) cur[x] += (x & 1) ? wo : we;
    for (int x = 1; x < 8; ++x)
      if (cur[x] > cur[best]) best = x;
    cur[best] -= c.len;
    c.xcd[i] = (uint8_t)best;
    c.before[i] = (uint16_t)c.count[best]++;
  }
  return c;
}
static_assert(kXcdWeightEven >= kXcdWeightOdd, "even XCDs take the larger share");
constexpr int kXcdCycleLen = make_xcd_cycle().len;
static_assert(kXcdCycleLen <= kXcdCycleMax, "XCD weights too fine for the cycle table");
static_assert(kXcdCycleMax <= kRankBuckets && kRankBuckets % 8 == 0,
              "the ordering kernel loads the cycle one entry per thread, fills queue t % 8");
__constant__ XcdCycle kXcdCycle = make_xcd_cycle();

// The dispatch order of an unchunked long-shard sweep, [8 * units_per_xcd] (workgroup index ->
// unit, -1 for none).  Workgroups are dispatched in index order, index i on XCD i % 8, and the
// long shards' workgroups live long, so
//  * the (request, shard) pairs are ranked by page count, longest first: a request's shards are
//    of one length, but across a ragged batch they differ 2x, and in shard-index order the last
//    units to start were full-length shards that streamed alone at the end of the launch
//    (longest-processing-time-first list scheduling);
//  * the ranked units (all KV heads of a pair in turn) are dealt to the 8 XCDs' queues in the
//    kXcdWeightEven : kXcdWeightOdd cycle, since the odd-numbered XCDs stream slower, when the
//    even XCDs' queues hold that many (else round-robin); the empty units and the padding fill
//    the rest of every queue.
// Measured on a ragged batch of 64 requests: ranking -4% step time, the weighted dealing -2.4%
// more.  Counting sort in one workgroup over kRankBuckets length buckets of 2^shift pages (the
// last bucket holds the empty shards only); pairs of one bucket keep no particular order among
// themselves.  The order decides only when and where a unit runs, never what it computes.
__global__ void __launch_bounds__(kRankBuckets)
rank_units_kernel(const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ n_shards,
                  int32_t batch, int32_t max_pages, int32_t max_shards, int32_t hkv,
                  int32_t units_per_xcd, int32_t shift, int32_t* __restrict__ unit_order) {
  __shared__ int32_t count[kRankBuckets];
  __shared__ int32_t scan[2][kRankBuckets];
  __shared__ int32_t ranked[kRankMaxPairs];  // pair index of rank r (unit order: r % B, S-1-r/B)
  __shared__ uint16_t key[kRankMaxPairs];    // bucket of pair r
  __shared__ uint8_t cyc_xcd[kXcdCycleMax];
  __shared__ uint16_t cyc_before[kXcdCycleMax];
  __shared__ int32_t cyc_count[8];
  __shared__ int32_t s_live;
  __shared__ int32_t used[8], first_free[8];
  const int t = threadIdx.x, lane = t & 63;
  const int n_pairs = batch * max_shards;
  constexpr int cycle = kXcdCycleLen;
  // x / hkv and x % hkv: a shift and a mask for the usual power-of-two head counts.
  const int hkv_log2 = (hkv & (hkv - 1)) == 0 ? __builtin_ctz(hkv) : -1;
  auto unit_of = [&](int rank, int j) {  // KV head j % hkv of the pair of rank rank + j / hkv
    return hkv_log2 >= 0 ? ranked[rank + (j >> hkv_log2)] * hkv + (j & (hkv - 1))
                         : ranked[rank + j / hkv] * hkv + j % hkv;
  };
  if (t < cycle) {
    cyc_xcd[t] = kXcdCycle.xcd[t];
    cyc_before[t] = kXcdCycle.before[t];
  }
  if (t < 8) {
    cyc_count[t] = kXcdCycle.count[t];
    used[t] = 0;
  }
  count[t] = 0;
  __syncthreads();
  // Every pair's bucket, kept and counted.  Most pairs of a ragged batch are empty (slots past a
  // request's shards): the empty bucket takes one atomic per wavefront.  (The loops run
  // uniformly over the workgroup, so every ballot sees whole wavefronts.)
  for (int r0 = 0; r0 < n_pairs; r0 += kRankBuckets) {
    const int r = r0 + t;
    int k = 0;
    if (r < n_pairs) {
      const ShardRange range = shard_range(ctx_lens, n_shards, r % batch,
                                           max_shards - 1 - r / batch, max_pages, max_shards);
      const int len = range.p1 - range.p0;
      k = len == 0 ? kRankBuckets - 1 : kRankBuckets - 2 - min(len >> shift, kRankBuckets - 2);
      key[r] = (uint16_t)k;
    }
    const bool empty = r < n_pairs && k == kRankBuckets - 1;
    const uint64_t m = __ballot(empty);
    if (r < n_pairs && !empty) atomicAdd(&count[k], 1);
    if (lane == 0 && m != 0) atomicAdd(&count[kRankBuckets - 1], (int)__popcll(m));
  }
  __syncthreads();
  if (t == 0) s_live = n_pairs - count[kRankBuckets - 1];
  // Exclusive prefix sums of the counts (Hillis-Steele over the shifted counts).
  int cur = 0;
  scan[0][t] = t > 0 ? count[t - 1] : 0;
  __syncthreads();
  for (int d = 1; d < kRankBuckets; d <<= 1) {
    scan[cur ^ 1][t] = scan[cur][t] + (t >= d ? scan[cur][t - d] : 0);
    cur ^= 1;
    __syncthreads();
  }
  count[t] = scan[cur][t];  // first rank of bucket t
  __syncthreads();
  for (int r0 = 0; r0 < n_pairs; r0 += kRankBuckets) {
    const int r = r0 + t;
    const int k = r < n_pairs ? key[r] : 0;
    const bool empty = r < n_pairs && k == kRankBuckets - 1;
    const uint64_t m = __ballot(empty);
    int base = 0;
    if (lane == 0 && m != 0) base = atomicAdd(&count[kRankBuckets - 1], (int)__popcll(m));
    base = __shfl(base, 0);
    if (r < n_pairs) {
      const int at = empty ? base + (int)__popcll(m & ((1ull << lane) - 1))
                           : atomicAdd(&count[k], 1);
      ranked[at] = r;
    }
  }
  __syncthreads();

  // Live unit k (k < R) is KV head k % hkv of the pair of rank k / hkv.  Its XCD and place in that
  // XCD's queue: entry k % cycle of the weighted cycle, or round-robin.
  const int R = s_live * hkv;
  const int full = R / cycle;
  const bool weighted = (int64_t)(full + 1) * cyc_count[0] <= units_per_xcd;
  if (weighted && t < R % cycle) atomicAdd(&used[cyc_xcd[t]], 1);
  __syncthreads();
  if (t < 8) used[t] += weighted ? full * cyc_count[t] : (R + 7 - t) / 8;
  __syncthreads();
  if (t == 0) {
    int acc = 0;
    for (int x = 0; x < 8; ++x) {
      first_free[x] = acc;
      acc += units_per_xcd - used[x];
    }
  }
  __syncthreads();
  for (int k = t; k < R; k += kRankBuckets) {
    int x, pos;
    if (weighted) {
      const int i = k % cycle;
      x = cyc_xcd[i];
      pos = (k / cycle) * cyc_count[x] + cyc_before[i];
    } else {
      x = k & 7;
      pos = k >> 3;
    }
    unit_order[8 * pos + x] = unit_of(0, k);
  }
  // The rest of every queue: empty unit e is KV head e % hkv of the pair of rank s_live + e / hkv
  // (then -1).  Thread t fills queue t % 8 (kRankBuckets is a multiple of 8), places
  // t / 8, t / 8 + 128, ... from the queue's first free one on.
  const int n_empty = n_pairs * hkv - R;
  const int x = t & 7;
  constexpr int kStride = kRankBuckets / 8;
  const int lo = used[x];
  int pos = t >> 3;
  if (pos < lo) pos += (lo - pos + kStride - 1) / kStride * kStride;
  for (int e = first_free[x] + pos - lo; pos < units_per_xcd; pos += kStride, e += kStride)
    unit_order[8 * pos + x] = e < n_empty ? unit_of(s_live, e) : -1;
}

// Fill p.unit_order (when the sweep has one) on `stream`, ahead of the sweep.
hipError_t launch_rank(const SplitParams& p, hipStream_t stream) {
  if (p.unit_order == nullptr) return hipSuccess;
  hipLaunchKernelGGL(rank_units_kernel, dim3(1), dim3(kRankBuckets), 0, stream, p.ctx_lens,
                     p.n_shards, p.batch, p.max_pages, p.max_shards, p.hkv, p.units_per_xcd,
                     p.rank_shift, p.unit_order);
  return hipGetLastError();
}

template <int G, int W, int NBUF>
__global__ void __launch_bounds__(64 * W)
__attribute__((amdgpu_waves_per_eu(G >= 8 ? 2 : 3)))   // the unfused sweep's occupancy
decode_fused_kernel(const uint16_t* __restrict__ qp, const uint16_t* __restrict__ kp,
                    const uint16_t* __restrict__ vp, const int32_t* __restrict__ block_table,
                    const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ n_shards,
                    float* __restrict__ out_o, float* __restrict__ out_lse, int32_t hq,
                    int32_t hkv, int32_t max_pages, int32_t num_pages, int32_t max_shards,
                    int32_t chunks, int32_t n_units, int32_t units_per_xcd, int32_t batch,
                    int32_t order, float scale_log2, int32_t* __restrict__ counters,
                    uint16_t* __restrict__ merged_o, float* __restrict__ merged_lse) {
  sweep_unit<G, W, NBUF, true>(qp, kp, vp, block_table, ctx_lens, n_shards, out_o, out_lse, hq,
                               hkv, max_pages, num_pages, max_shards, chunks, n_units,
                               units_per_xcd, batch, order, scale_log2, blockIdx.x, counters,
                               merged_o, merged_lse);
}

template <int G>
hipError_t launch_fused_g(const SplitParams& p, int32_t* counters, void* out, float* lse,
                          hipStream_t stream) {
  const unsigned grid = 8u * (unsigned)p.units_per_xcd;
  hipLaunchKernelGGL((decode_fused_kernel<G, kSplitWaves, kSplitBuffers>), dim3(grid),
                     dim3(64 * kSplitWaves), 0, stream, p.q, p.k, p.v, p.block_table, p.ctx_lens,
                     p.n_shards, p.out_o, p.out_lse, p.hq, p.hkv, p.max_pages, p.num_pages,
                     p.max_shards, p.chunks, p.n_units, p.units_per_xcd, p.batch, p.order,
                     p.scale_log2, counters, static_cast<uint16_t*>(out), lse);
  return hipGetLastError();
}

template <int G, int NBUF>
hipError_t launch_gn(const SplitParams& p, hipStream_t stream) {
  const hipError_t e = launch_rank(p, stream);
  if (e != hipSuccess) return e;
  const unsigned grid = 8u * (unsigned)p.units_per_xcd;
  hipLaunchKernelGGL((decode_split_kernel<G, kSplitWaves, NBUF>), dim3(grid), dim3(64 * kSplitWaves),
                     0, stream, p.q, p.k, p.v, p.block_table, p.ctx_lens, p.n_shards, p.out_o,
                     p.out_lse, p.hq, p.hkv, p.max_pages, p.num_pages, p.max_shards, p.chunks,
                     p.n_units, p.units_per_xcd, p.batch, p.order, p.scale_log2, p.unit_order);
  return hipGetLastError();
}

// The host picks deep buffers from the shard length (short shards of at least kDeepMinPages);
// NBUF only changes how far ahead pages are requested, never the arithmetic.
template <int G>
hipError_t launch_g(const SplitParams& p, hipStream_t stream) {
  if (p.deep) return launch_gn<G, split_buffers_deep(G)>(p, stream);
  return launch_gn<G, kSplitBuffers>(p, stream);
}

// One launch, two roles: the sweep's workgroups and those of a fused product (linear_body.h) share
// one grid, so the hardware dispatcher runs both at once on every CU (the sweep beside the
// feed-forward, §3).  Groups of 8 consecutive workgroup indices (one per XCD) are dealt to the two
// roles in proportion to their sizes, so both start together and each keeps its index modulo 8;
// every workgroup does exactly what it would do in its own launch.
// The occupancy the sweep alone reaches (registers), asked of the shared kernel too, so that
// the product's role does not lower it.
template <int G, int MB>
__global__ void __launch_bounds__(64 * kSplitWaves)
__attribute__((amdgpu_waves_per_eu(G >= 8 ? 2 : 3)))
sweep_beside_linear_kernel(
    const uint16_t* __restrict__ qp, const uint16_t* __restrict__ kp,
    const uint16_t* __restrict__ vp, const int32_t* __restrict__ block_table,
    const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ n_shards,
    float* __restrict__ out_o, float* __restrict__ out_lse, int32_t hq, int32_t hkv,
    int32_t max_pages, int32_t num_pages, int32_t max_shards, int32_t chunks, int32_t n_units,
    int32_t units_per_xcd, int32_t batch, int32_t order, float scale_log2,
    const int32_t* __restrict__ unit_order, const uint16_t* __restrict__ x,
    const uint16_t* __restrict__ w,
    const uint16_t* __restrict__ gain, const uint16_t* __restrict__ residual,
    uint16_t* __restrict__ out_a, uint16_t* __restrict__ out_b, int32_t M, int32_t N, int32_t K,
    int32_t n_split, float eps, int32_t prologue, int32_t glu, int32_t linear_groups) {
  static_assert(64 * kSplitWaves == lin::kThreads, "both roles use the same workgroup size");
  const unsigned j = blockIdx.x / 8u, lane8 = blockIdx.x % 8u;
  const unsigned long long S = (unsigned)units_per_xcd, T = S + (unsigned)linear_groups;
  const unsigned before = (unsigned)(j * S / T);          // sweep groups dealt before group j
  if ((unsigned)((j + 1ull) * S / T) > before) {
    sweep_unit<G, kSplitWaves, kSplitBuffers>(qp, kp, vp, block_table, ctx_lens, n_shards, out_o,
                                              out_lse, hq, hkv, max_pages, num_pages, max_shards,
                                              chunks, n_units, units_per_xcd, batch, order,
                                              scale_log2, 8u * before + lane8, nullptr, nullptr,
                                              nullptr, unit_order);
    return;
  }
  constexpr int U = 2, R = lin::beside_rows(MB), RG = lin::beside_rows_glu(MB);
  const unsigned lb = 8u * (j - before) + lane8;
  if (glu) {
    if (prologue == kProRmsNorm)
      lin::linear_rows<kProRmsNorm, MB, U, RG, true>(x, w, gain, residual, out_a, out_b, M, N, K,
                                                     n_split, eps, lb);
    else
      lin::linear_rows<kProNone, MB, U, RG, true>(x, w, gain, residual, out_a, out_b, M, N, K,
                                                  n_split, eps, lb);
    return;
  }
  if (prologue == kProRmsNorm)
    lin::linear_rows<kProRmsNorm, MB, U, R>(x, w, gain, residual, out_a, out_b, M, N, K, n_split,
                                            eps, lb);
  else if (prologue == kProSwiglu)
    lin::linear_rows<kProSwiglu, MB, U, R>(x, w, gain, residual, out_a, out_b, M, N, K, n_split,
                                           eps, lb);
  else
    lin::linear_rows<kProNone, MB, U, R>(x, w, gain, residual, out_a, out_b, M, N, K, n_split,
                                         eps, lb);
}

template <int G, int MB>
hipError_t launch_beside(const SplitParams& p, const LinearParams& l, hipStream_t stream) {
  const int rows = l.glu ? lin::beside_rows_glu(MB) : lin::beside_rows(MB);
  const int linear_groups = (lin::linear_blocks(l.N, rows) + 7) / 8;
  const unsigned grid = 8u * ((unsigned)p.units_per_xcd + (unsigned)linear_groups);
  const hipError_t e = launch_rank(p, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((sweep_beside_linear_kernel<G, MB>), dim3(grid), dim3(64 * kSplitWaves), 0,
                     stream, p.q, p.k, p.v, p.block_table, p.ctx_lens, p.n_shards, p.out_o,
                     p.out_lse, p.hq, p.hkv, p.max_pages, p.num_pages, p.max_shards, p.chunks,
                     p.n_units, p.units_per_xcd, p.batch, p.order, p.scale_log2, p.unit_order,
                     l.x, l.w, l.gain,
                     l.residual, l.out_a, l.out_b, l.M, l.N, l.K, l.n_split, l.eps, l.prologue,
                     l.glu ? 1 : 0, linear_groups);
  return hipGetLastError();
}

template <int G>
hipError_t launch_beside_g(const SplitParams& p, const LinearParams& l, hipStream_t stream) {
  switch (lin::rows_bucket(l.M)) {
    case 1: return launch_beside<G, 1>(p, l, stream);
    case 2: return launch_beside<G, 2>(p, l, stream);
    case 4: return launch_beside<G, 4>(p, l, stream);
    default: return launch_beside<G, 8>(p, l, stream);
  }
}

template <int G>
int resident_g() {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per_cu, decode_split_kernel<G, kSplitWaves, kSplitBuffers>, 64 * kSplitWaves, 0) !=
          hipSuccess) {
    (void)hipGetLastError();  // leave no error behind for the next launch check
    return 0;
  }
  return cus * per_cu;
}

}  // namespace

int split_resident_workgroups(int group) {
  static std::atomic<int> cached[4] = {{-1}, {-1}, {-1}, {-1}};
  const int k = group == 1 ? 0 : group == 2 ? 1 : group == 4 ? 2 : group == 8 ? 3 : -1;
  if (k < 0) return 0;
  int v = cached[k].load(std::memory_order_relaxed);
  if (v < 0) {
    v = k == 0 ? resident_g<1>() : k == 1 ? resident_g<2>() : k == 2 ? resident_g<4>() : resident_g<8>();
    if (v > 0) cached[k].store(v, std::memory_order_relaxed);
  }
  return v;
}

hipError_t launch_decode_split(const SplitParams& p, int group, hipStream_t stream) {
  switch (group) {
    case 1: return launch_g<1>(p, stream);
    case 2: return launch_g<2>(p, stream);
    case 4: return launch_g<4>(p, stream);
    case 8: return launch_g<8>(p, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_decode_split_beside(const SplitParams& p, int group, const LinearParams& l,
                                     hipStream_t stream) {
  switch (group) {
    case 1: return launch_beside_g<1>(p, l, stream);
    case 2: return launch_beside_g<2>(p, l, stream);
    case 4: return launch_beside_g<4>(p, l, stream);
    case 8: return launch_beside_g<8>(p, l, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_decode_fused(const SplitParams& p, int group, int32_t* counters, void* out,
                               float* lse, hipStream_t stream) {
  switch (group) {
    case 1: return launch_fused_g<1>(p, counters, out, lse, stream);
    case 2: return launch_fused_g<2>(p, counters, out, lse, stream);
    case 4: return launch_fused_g<4>(p, counters, out, lse, stream);
    case 8: return launch_fused_g<8>(p, counters, out, lse, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace qf
