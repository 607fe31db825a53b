// Paged cache append of the current token (Q-First, arXiv:2608.15473, §2): one workgroup per
// request runs the append body of append_body.h.
#include "append_body.h"

namespace qf {
namespace {

__global__ void __launch_bounds__(256)
kv_append_kernel(uint16_t* __restrict__ k, uint16_t* __restrict__ v,
                 const int32_t* __restrict__ block_table, int32_t* __restrict__ ctx_lens,
                 const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
                 int32_t* __restrict__ status, int32_t hkv, int32_t max_pages, int32_t num_pages,
                 int32_t advance) {
  app::append_request(k, v, block_table, ctx_lens, k_new, v_new, status, hkv, max_pages, num_pages,
                      advance, blockIdx.x);
}

}  // namespace

hipError_t launch_kv_append(const AppendParams& p, hipStream_t stream) {
  if (p.batch == 0) return hipSuccess;
  hipLaunchKernelGGL(kv_append_kernel, dim3(p.batch), dim3(256), 0, stream, p.k, p.v,
                     p.block_table, p.ctx_lens, p.k_new, p.v_new, p.status, p.hkv, p.max_pages,
                     p.num_pages, p.advance);
  return hipGetLastError();
}

}  // namespace qf
