// Internal interface between the host library (qfattn_api.hip) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qf {

constexpr int kHeadDim = 128;     // D
constexpr int kPage = 16;         // P
constexpr int kSplitWaves = 4;    // waves per workgroup of the sweep kernel
// Pages in registers per wave of the sweep (1 computed, the rest in flight).  Long shards keep
// three wavefronts per SIMD with 2.  Short shards of some length (a handful of pages per
// wavefront, so a workgroup's life is mostly its first pages' latency) go deeper, at two
// wavefronts per SIMD: measured on MI355X, 5 buffers make 32-page shards at G=2 2% faster, while
// long ragged shards lose 4% at that occupancy and shards of 2-3 pages per wavefront lose up to
// 19% (the occupancy is lost and the extra buffers stay empty).
constexpr int kSplitBuffers = 2;
constexpr int split_buffers_deep(int group) { return group <= 2 ? 5 : group == 4 ? 3 : 2; }
constexpr int kDeepMinPages = 4 * kSplitWaves;   // shard pages (at full capacity) for deep buffers

// Dispatch orders of the sweep's units (see decode_split.hip).
constexpr int kOrderByRequest = 0;
constexpr int kOrderByShardDesc = 1;
// Shards at least this long (pages, at full capacity) are swept in kOrderByShardDesc.
constexpr int kLongShardPages = 128;
// Relative page shares of the sub-shard chunks of a long shard that run on even- and odd-numbered
// XCDs (decode_split.hip): the odd XCDs stream slower.
constexpr int kXcdWeightEven = 1080;
constexpr int kXcdWeightOdd = 920;
// The one-workgroup kernel that orders the units of an unchunked long-shard sweep
// (decode_split.hip): length buckets (= its threads), and the most (request, shard) pairs it
// ranks (held in LDS).
constexpr int kRankBuckets = 1024;
constexpr int kRankMaxPairs = 8192;

// One launch of the sweep kernel.  A workgroup handles one unit (request b, shard s, chunk c,
// KV head g); its output slot is [((b * max_shards + s) * chunks + c) * hq + g * G + h].
struct SplitParams {
  const uint16_t* q;            // bf16 [B, Hq, D]
  const uint16_t* k;            // bf16 [num_pages, Hkv, P, D]
  const uint16_t* v;
  const int32_t* block_table;   // [B, max_pages] or null (identity)
  const int32_t* ctx_lens;      // [B]
  const int32_t* n_shards;      // [B]
  float* out_o;                 // fp32 [B, max_shards, chunks, Hq, D]
  float* out_lse;               // fp32 [B, max_shards, chunks, Hq]
  int32_t batch, hq, hkv, max_pages, num_pages, max_shards, chunks;
  int32_t n_units;              // B * max_shards * chunks * Hkv
  int32_t units_per_xcd;        // ceil(n_units / 8)
  int32_t order;                // kOrderByRequest or kOrderByShardDesc (dispatch order of units)
  // kOrderByShardDesc with chunks == 1 only, or null: [8 * units_per_xcd] int32 that an ordering
  // kernel, launched just before the sweep, fills with the unit each workgroup index sweeps (-1:
  // none): longest shard first, dealt to the XCDs by kXcdWeightEven / kXcdWeightOdd
  // (rank_shift: log2 of the length buckets' width in pages).
  int32_t* unit_order;
  int32_t rank_shift;
  bool deep;                    // short shards of >= kDeepMinPages pages: split_buffers_deep(G)
  float scale_log2;             // softmax scale * log2(e)
};

// Merge of `entries` partial states per (row, head):
//   in  O [rows, entries, hq, D] fp32, lse [rows, entries, hq] fp32 (natural log)
//   out O [rows, hq, D] (fp32 or bf16), lse [rows, hq] fp32 (may be null)
// With q non-null (final output only) the current token is folded in after the merge:
//   q bf16 [rows, hq, D], k_cur / v_cur bf16 [rows, hkv, D].
struct AppendParams;

struct MergeParams {
  const float* in_o;
  const float* in_lse;
  void* out_o;
  float* out_lse;
  int32_t rows, entries, hq;
  const uint16_t* q = nullptr;
  const uint16_t* k_cur = nullptr;
  const uint16_t* v_cur = nullptr;
  int32_t hkv = 1;
  float scale = 0.0f;
  // With the current token (q, k_cur, v_cur): also append k_cur and v_cur to the cache and
  // advance ctx_lens (AppendParams below; k_new / v_new / advance there are not used).
  const AppendParams* append = nullptr;
};

// Cache append: write the current token's key and value at position ctx_lens[b] of request b.
struct AppendParams {
  uint16_t* k;                  // bf16 [num_pages, Hkv, P, D]
  uint16_t* v;
  const int32_t* block_table;   // [B, max_pages] or null (identity)
  int32_t* ctx_lens;            // [B]; advanced by one after the write when advance != 0
  const uint16_t* k_new;        // bf16 [B, Hkv, D]
  const uint16_t* v_new;
  int32_t* status;              // optional: set to 1 when an append is skipped
  int32_t batch, hkv, max_pages, num_pages, advance;
};

hipError_t launch_kv_append(const AppendParams& p, hipStream_t stream);
// out = W . P(x) (+ residual) for a few input rows (block_ops.hip).
constexpr int kProNone = 0, kProRmsNorm = 1, kProSwiglu = 2;
constexpr int kLinearMaxRows = 8;
struct LinearParams {
  const uint16_t* x;         // bf16 [M, K] ([M, 2K] for kProSwiglu: gate, then up)
  const uint16_t* w;         // bf16 [N, K]
  const uint16_t* gain;      // bf16 [K] (kProRmsNorm)
  const uint16_t* residual;  // bf16 [M, N] or nullptr
  uint16_t* out_a;           // bf16 [M, n_split]
  uint16_t* out_b;           // bf16 [M, N - n_split]
  int M, N, K, n_split, prologue;
  float eps;
  bool glu;                  // rows of W alternate gate / up; out = silu(gate) * up, N / 2 columns
};
hipError_t launch_linear(const LinearParams& p, hipStream_t stream);
// The sweep with the merge fused into its last workgroup per (request, KV head)
// (decode_split.hip): p.out_o / p.out_lse hold the partial states, counters [batch * hkv] int32
// start at zero and are left at zero.
hipError_t launch_decode_fused(const SplitParams& p, int group, int32_t* counters, void* out,
                               float* lse, hipStream_t stream);
// The sweep and a fused product in one launch (decode_split.hip).
hipError_t launch_decode_split_beside(const SplitParams& p, int group, const LinearParams& l,
                                      hipStream_t stream);

// Host simulation of the layer-wise decode schedule (schedule.cpp).
int simulate_schedule(int R, const double* arrival, const double* attn_time, int L, int wiring,
                      double ffn_time, int min_batch, double max_wait, double* finish,
                      double* sweep_start, double* sweep_end, double* ffn_depart,
                      double* ffn_return);

hipError_t launch_decode_split(const SplitParams& p, int group, hipStream_t stream);

// The allocation-free decode's fixed scratch (decode_noalloc.hip): one device array per GPU of
// kNoallocScratchBytes, the counters in its first kNoallocCounterBytes, the partial states after.
constexpr size_t kNoallocScratchBytes = size_t(64) << 20;
constexpr size_t kNoallocCounterBytes = size_t(256) << 10;
constexpr size_t kNoallocStateBytes = kNoallocScratchBytes - kNoallocCounterBytes;
// This device's scratch (looked up on the first call on the device): *counters (n_counters int32
// entries, cleared to zero on `stream` before anything else is enqueued there) and *states.
hipError_t noalloc_prepare(int32_t n_counters, hipStream_t stream, int32_t** counters,
                           void** states);

// Workgroups of the long-shard sweep (kSplitBuffers) at group size `group` that are resident on
// the current device at once (compute units x workgroups per unit); 0 when there is no device to
// ask.  Queried once per group size and kept.
int split_resident_workgroups(int group);
// to_bf16 = false: partial-state output (fp32 O not written for an empty row);
// to_bf16 = true:  final output (bf16, +0 for an empty row).
hipError_t launch_merge(const MergeParams& p, bool to_bf16, hipStream_t stream);

}  // namespace qf
