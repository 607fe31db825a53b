// Merge kernels: partial softmax states of shards (or of a shard's chunks) into one (Q-First,
// arXiv:2608.15473, §5), optionally followed by the current token (§2, Appendix A).  The body
// is in merge_body.h.
#include "append_body.h"
#include "merge_body.h"

namespace qf {
namespace {

// W wavefronts per workgroup, each taking 16 slots per round: as many as one round needs, up to 16
// (rows of more than 256 slots take more rounds).
template <bool BF16, bool CUR, int W>
__global__ void __launch_bounds__(64 * W)
merge_kernel(const float* __restrict__ in_o, const float* __restrict__ in_lse,
             void* __restrict__ out_o, float* __restrict__ out_lse, int32_t entries,
             int32_t hq, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cur,
             const uint16_t* __restrict__ v_cur, int32_t hkv, float scale) {
  mrg::merge_row<BF16, CUR, W>(in_o, in_lse, out_o, out_lse, entries, hq, blockIdx.x / hq,
                               blockIdx.x % hq, q, k_cur, v_cur, hkv, scale);
}

// The merge with the current token and the current token's cache append in one launch: the first
// rows * hq workgroups merge (request b, query head h); each of the last `rows` workgroups writes
// k_j and v_j of every KV head of its request at position ctx_lens[b] and advances it, at the same
// time.  No other workgroup of the launch reads ctx_lens or the cache, and the sweep that produced
// the partials never reads position ctx_lens[b], so the write races with nothing.
template <int W>
__global__ void __launch_bounds__(64 * W)
merge_append_kernel(const float* __restrict__ in_o, const float* __restrict__ in_lse,
                    void* __restrict__ out_o, float* __restrict__ out_lse, int32_t entries,
                    int32_t hq, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cur,
                    const uint16_t* __restrict__ v_cur, int32_t hkv, float scale,
                    uint16_t* __restrict__ k_cache, uint16_t* __restrict__ v_cache,
                    const int32_t* __restrict__ block_table, int32_t* __restrict__ ctx_lens,
                    int32_t* __restrict__ status, int32_t max_pages, int32_t num_pages,
                    int32_t merge_blocks) {
  if ((int)blockIdx.x >= merge_blocks) {
    app::append_request(k_cache, v_cache, block_table, ctx_lens, k_cur, v_cur, status, hkv,
                        max_pages, num_pages, 1, (int)blockIdx.x - merge_blocks);
    return;
  }
  mrg::merge_row<true, true, W>(in_o, in_lse, out_o, out_lse, entries, hq, blockIdx.x / hq,
                                blockIdx.x % hq, q, k_cur, v_cur, hkv, scale);
}

template <int W>
hipError_t launch_w(const MergeParams& p, bool to_bf16, unsigned grid, hipStream_t stream) {
  if (p.append) {
    const AppendParams& a = *p.append;
    hipLaunchKernelGGL((merge_append_kernel<W>), dim3(grid + (unsigned)p.rows), dim3(64 * W), 0,
                       stream, p.in_o, p.in_lse, p.out_o, p.out_lse, p.entries, p.hq, p.q, p.k_cur,
                       p.v_cur, p.hkv, p.scale, a.k, a.v, a.block_table, a.ctx_lens, a.status,
                       a.max_pages, a.num_pages, (int32_t)grid);
    return hipGetLastError();
  }
  if (p.q)
    hipLaunchKernelGGL((merge_kernel<true, true, W>), dim3(grid), dim3(64 * W), 0, stream, p.in_o,
                       p.in_lse, p.out_o, p.out_lse, p.entries, p.hq, p.q, p.k_cur, p.v_cur,
                       p.hkv, p.scale);
  else if (to_bf16)
    hipLaunchKernelGGL((merge_kernel<true, false, W>), dim3(grid), dim3(64 * W), 0, stream,
                       p.in_o, p.in_lse, p.out_o, p.out_lse, p.entries, p.hq, nullptr, nullptr,
                       nullptr, 1, 0.0f);
  else
    hipLaunchKernelGGL((merge_kernel<false, false, W>), dim3(grid), dim3(64 * W), 0, stream,
                       p.in_o, p.in_lse, p.out_o, p.out_lse, p.entries, p.hq, nullptr, nullptr,
                       nullptr, 1, 0.0f);
  return hipGetLastError();
}

}  // namespace

// The workgroup of a row has just the wavefronts its slots need (16 slots each): measured on MI355X,
// 2 wavefronts instead of 4 for 24 slots made the 4,608-position single layer's step 3% faster,
// and 8 instead of 16 for 96 slots the per-GPU share of the 2^20-token request's 0.5%.  The result
// does not depend on W as long as one round suffices: every wavefront sums the same 16 slots, and
// the wavefronts without slots add exact zeros in the cross-wavefront merge.
hipError_t launch_merge(const MergeParams& p, bool to_bf16, hipStream_t stream) {
  const unsigned grid = (unsigned)p.rows * (unsigned)p.hq;
  if (grid == 0) return hipSuccess;
  if (p.entries > 128) return launch_w<16>(p, to_bf16, grid, stream);
  if (p.entries > 64) return launch_w<8>(p, to_bf16, grid, stream);
  if (p.entries > 32) return launch_w<4>(p, to_bf16, grid, stream);
  if (p.entries > 16) return launch_w<2>(p, to_bf16, grid, stream);
  return launch_w<1>(p, to_bf16, grid, stream);
}

}  // namespace qf
