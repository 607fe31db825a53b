// Merge of partial softmax states (O_i, ln Z_i) (Q-First, arXiv:2608.15473, §5).
//
// For one (row, query head) and entries i = 0..N-1:
//   m = max_i ln Z_i,   w_i = exp(ln Z_i - m),   out = sum_i w_i O_i / sum_i w_i,
//   ln Z = m + ln(sum_i w_i).
// This is the pairwise lerp/sigmoid/logaddexp merge of §5 applied to all entries at once; every
// weight is <= 1, so it is finite for any magnitude of the log partitions.  An entry with
// ln Z = -inf is empty: its weight is selected to 0 and its O (possibly garbage, §5) is never
// multiplied.  A NaN among the ln Z makes the row's output NaN.
//
// One workgroup per (row, head); its wavefronts take the entries in groups of 16, and the
// wavefronts' sums meet in LDS.  Within a group the entries lie across the lanes (lane k holds
// entry k's ln Z, so one exponential and a 16-lane reduction serve all 16) and each lane sums its
// own 2 of the 128 dims over the group's O rows.  The body is shared by the merge kernels and by
// the sweep's last workgroup of a (request, KV head) when the two are fused.
//
// With the current token (CUR): the merged pair is the cache's (o_<j, lse_<j), and the current
// token is folded in as §2 and Appendix A state it: s_jj = scale * q_j . k_j,
// out = lerp(v_j, o_<j, sigma(lse_<j - s_jj)) with sigma(x) = 1 / (1 + exp(-x)), and
// lse = logaddexp(lse_<j, s_jj).  An empty cache gives sigma(-inf) = 0, i.e. out = v_j.
#pragma once

#include <math.h>

#include "qf_internal.h"

namespace qf {
namespace mrg {

constexpr int D = kHeadDim;

// fp32 -> bf16, round to nearest even; NaN stays a (quiet) NaN.
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x0040u;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Sum and maximum over the 16 lanes of a DPP row; the result is bitwise identical on all 16 lanes.
__device__ __forceinline__ float row_sum16(float x) {
  x += __builtin_amdgcn_update_dpp(0.0f, x, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
  x += __builtin_amdgcn_update_dpp(0.0f, x, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
  x += __builtin_amdgcn_update_dpp(0.0f, x, 0x141, 0xF, 0xF, false);  // row_half_mirror
  x += __builtin_amdgcn_update_dpp(0.0f, x, 0x140, 0xF, 0xF, false);  // row_mirror
  return x;
}

__device__ __forceinline__ float row_max16(float x) {
  x = fmaxf(x, __builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false));
  x = fmaxf(x, __builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false));
  x = fmaxf(x, __builtin_amdgcn_update_dpp(x, x, 0x141, 0xF, 0xF, false));
  x = fmaxf(x, __builtin_amdgcn_update_dpp(x, x, 0x140, 0xF, 0xF, false));
  return x;
}

// Lane k's value, as a wavefront-uniform scalar.
__device__ __forceinline__ float lane_value(float x, int k) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), k));
}

constexpr int K = 16;  // entries per wavefront and round

// A wavefront's running merge: its maximum m, the weight sum L and, per lane, the weighted sum of
// the lane's two dims (every weight exp(ln Z_i - m) <= 1), and whether a ln Z was NaN.
struct WaveMerge {
  float m = -INFINITY;
  float L = 0.0f;
  float2 acc = make_float2(0.0f, 0.0f);
  bool nan = false;

  // Adds a group of up to K entries: lane k < K holds entry k's ln Z in x (-inf for an empty or
  // absent entry, and in lanes K..63), v[k] entry k's O at this lane's dims.  An entry with weight
  // 0 (empty, or too far below the maximum for fp32) is selected out: its O, which may be garbage,
  // is never multiplied.  The maximum only grows; the sums are rescaled when it does.
  __device__ __forceinline__ void add(float x, const float2 (&v)[K]) {
    nan |= __ballot(x != x) != 0;
    const float mc = fmaxf(m, lane_value(row_max16(x), 0));
    if (mc == -INFINITY) return;  // nothing live so far
    const float f = (m == -INFINITY) ? 0.0f : expf(m - mc);
    m = mc;
    const float w = (x == -INFINITY) ? 0.0f : expf(x - mc);
    L = fmaf(L, f, lane_value(row_sum16(w), 0));
    acc.x *= f;
    acc.y *= f;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const float wk = lane_value(w, k);
      if (wk != 0.0f) {
        acc.x = fmaf(wk, v[k].x, acc.x);
        acc.y = fmaf(wk, v[k].y, acc.y);
      }
    }
  }
};

// The LDS meeting point of W wavefronts' merges.
template <int W>
struct WaveMergeLds {
  float2 acc[W][64];
  float L[W];
  float m[W];
  int nan[W];

  __device__ __forceinline__ void put(int wave, int lane, const WaveMerge& s) {
    acc[wave][lane] = s.acc;
    if (lane == 0) {
      L[wave] = s.L;
      m[wave] = s.m;
      nan[wave] = s.nan;
    }
  }

  // Wavefronts w0 .. w0+n-1 (n <= 16) merged, read by one whole wavefront: the normalised output
  // pair of this lane's dims and ln Z, NaN if any ln Z was NaN, (0, -inf) if every entry was
  // empty.  Wavefronts without entries add exact zeros, so the result does not depend on how many
  // of them there are.
  __device__ __forceinline__ float2 finish(int w0, int n, int lane, float& lse_out) const {
    const bool in = lane < n;
    const float mw = in ? m[w0 + lane] : -INFINITY;
    const bool any_nan = __ballot(in && nan[w0 + lane] != 0) != 0;
    const float M = lane_value(row_max16(mw), 0);
    const float f = (mw == -INFINITY) ? 0.0f : expf(mw - M);
    const float Lt = lane_value(row_sum16(in ? f * L[w0 + lane] : 0.0f), 0);
    float2 a = make_float2(0.0f, 0.0f);
    for (int w = 0; w < n; ++w) {
      const float fw = lane_value(f, w);
      a.x = fmaf(fw, acc[w0 + w][lane].x, a.x);
      a.y = fmaf(fw, acc[w0 + w][lane].y, a.y);
    }
    if (any_nan) {
      lse_out = NAN;
      return make_float2(NAN, NAN);
    }
    if (M == -INFINITY) {
      lse_out = -INFINITY;
      return make_float2(0.0f, 0.0f);
    }
    lse_out = M + logf(Lt);
    return make_float2(a.x / Lt, a.y / Lt);
  }
};

// Row r (request, or request x shard for a chunk merge), query head h of the partial states
// in_o [rows, entries, hq, D], in_lse [rows, entries, hq]: merged into out_o / out_lse, then (CUR)
// the current token folded in.  Called by every thread of a workgroup of W <= 16 wavefronts.
// COHERENT: the partial states were written by other workgroups of the same launch (with
// device-scope stores), so they are read with device-scope loads, which bypass the XCD's
// non-coherent L2.
template <bool BF16, bool CUR, int W, bool COHERENT = false>
__device__ __forceinline__ void merge_row(
    const float* __restrict__ in_o, const float* __restrict__ in_lse, void* __restrict__ out_o,
    float* __restrict__ out_lse, int32_t entries, int32_t hq, const int r, const int h,
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cur,
    const uint16_t* __restrict__ v_cur, int32_t hkv, float scale) {
  static_assert(W >= 1 && W <= 16, "the wavefronts' merge takes one DPP row");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const float* lse = in_lse + (size_t)r * entries * hq + h;
  const float* o = in_o + ((size_t)r * entries * hq + h) * D;
  const int32_t o_step = hq * D;  // floats between entries

  // Wavefront w takes entries [K w, K w + K) of every K W: their log-partitions first (lane k
  // loads entry k's), then the O rows of the live ones among them, all loaded before any is used.
  // (Loading every O row together with the log-partitions, one round trip instead of two, was
  // measured no faster on MI355X, also where every entry is live; most slots of a ragged batch
  // are empty, and their O, never written, is not worth a read.)
  WaveMerge st;
  for (int i0 = K * wave; i0 < entries; i0 += K * W) {
    const int n = min(K, entries - i0);
    float x = -INFINITY;
    if (lane < n) {
      const float* p = &lse[(size_t)(i0 + lane) * hq];
      x = COHERENT ? __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : *p;
    }
    const uint64_t live = __ballot(x != -INFINITY);
    // Entry i0 + k's O pair at a 32-bit byte offset from one wavefront-uniform base (the offsets
    // of a round stay below K * hq * D * 4 bytes).
    const char* o_i0 = reinterpret_cast<const char*>(o + (size_t)i0 * o_step);
    float2 v[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      v[k] = make_float2(0.0f, 0.0f);
      if ((live >> k) & 1) {
        const float* p = reinterpret_cast<const float*>(o_i0 + (uint32_t)(lane * 8 + k * o_step * 4));
        if (COHERENT) {
          v[k].x = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          v[k].y = __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
          v[k] = *reinterpret_cast<const float2*>(p);
        }
      }
    }
    st.add(x, v);
  }

  __shared__ WaveMergeLds<W> lds;
  lds.put(wave, lane, st);
  __syncthreads();
  if (wave == 0) {
    float lse_out;
    float2 a = lds.finish(0, W, lane, lse_out);
    const bool empty = lse_out == -INFINITY;
    const size_t out_idx = ((size_t)r * hq + h) * D / 2 + lane;  // float2 / bf16-pair index
    if (CUR) {
      const int g = h / (hq / hkv);
      const uint32_t qw = reinterpret_cast<const uint32_t*>(q + ((size_t)r * hq + h) * D)[lane];
      const uint32_t kw = reinterpret_cast<const uint32_t*>(k_cur + ((size_t)r * hkv + g) * D)[lane];
      const uint32_t vw = reinterpret_cast<const uint32_t*>(v_cur + ((size_t)r * hkv + g) * D)[lane];
      float dot = fmaf(bf16_lo(qw), bf16_lo(kw), bf16_hi(qw) * bf16_hi(kw));
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) dot += __shfl_xor(dot, o);
      const float s_jj = dot * scale;
      const float t = 1.0f / (1.0f + expf(-(lse_out - s_jj)));   // weight of the cached history
      a.x = (1.0f - t) * bf16_lo(vw) + t * a.x;
      a.y = (1.0f - t) * bf16_hi(vw) + t * a.y;
      const float mx = fmaxf(lse_out, s_jj);
      float joined = mx + log1pf(expf(-fabsf(lse_out - s_jj)));  // stabilised logaddexp
      if (mx == -INFINITY) joined = -INFINITY;
      lse_out = (lse_out != lse_out || s_jj != s_jj) ? NAN : joined;
    }
    if (BF16) {
      reinterpret_cast<uint32_t*>(out_o)[out_idx] = bf16_rne(a.x) | (bf16_rne(a.y) << 16);
    } else if (!empty) {
      reinterpret_cast<float2*>(out_o)[out_idx] = a;
    }
    if (out_lse && lane == 0) out_lse[(size_t)r * hq + h] = lse_out;
  }
  __syncthreads();  // the LDS may be reused by a next call in the same workgroup
}

}  // namespace mrg
}  // namespace qf
