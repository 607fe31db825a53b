// Standalone launch of the fused decode-block products (body in linear_body.h).
#include "linear_body.h"

namespace qf {
namespace {

template <int PRO, int MB, int U, int R, bool GLU>
__global__ void __launch_bounds__(lin::kThreads)
linear_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
              const uint16_t* __restrict__ gain, const uint16_t* __restrict__ residual,
              uint16_t* __restrict__ out_a, uint16_t* __restrict__ out_b, int32_t M, int32_t N,
              int32_t K, int32_t n_split, float eps) {
  lin::linear_rows<PRO, MB, U, R, GLU>(x, w, gain, residual, out_a, out_b, M, N, K, n_split,
                                       eps, blockIdx.x);
}

// One row per wavefront; two (a gate row and its up row) with the GLU output.
template <int PRO, int MB, int U>
void launch_u(const LinearParams& p, hipStream_t stream) {
  if constexpr (PRO != kProSwiglu) {   // the host rejects a GLU output after a SwiGLU input
    if (p.glu) {
      hipLaunchKernelGGL((linear_kernel<PRO, MB, U, 2, true>), dim3(lin::linear_blocks(p.N, 2)),
                         dim3(lin::kThreads), 0, stream, p.x, p.w, p.gain, p.residual, p.out_a,
                         p.out_b, p.M, p.N, p.K, p.n_split, p.eps);
      return;
    }
  }
  hipLaunchKernelGGL((linear_kernel<PRO, MB, U, 1, false>), dim3(lin::linear_blocks(p.N, 1)),
                     dim3(lin::kThreads), 0, stream, p.x, p.w, p.gain, p.residual, p.out_a,
                     p.out_b, p.M, p.N, p.K, p.n_split, p.eps);
}

template <int PRO, int MB>
void launch_pro(const LinearParams& p, hipStream_t stream) {
  constexpr int cap = (MB <= 1) ? 8 : (MB <= 2) ? 4 : (MB <= 4) ? 2 : 1;
  switch (lin::pick_unroll(p.M, p.K)) {
    case 1: launch_u<PRO, MB, 1>(p, stream); break;
    case 2: launch_u<PRO, MB, (cap >= 2 ? 2 : 1)>(p, stream); break;
    case 4: launch_u<PRO, MB, (cap >= 4 ? 4 : 1)>(p, stream); break;
    default: launch_u<PRO, MB, (cap >= 8 ? 8 : 1)>(p, stream); break;
  }
}

template <int PRO>
void launch_rows(const LinearParams& p, hipStream_t stream) {
  switch (lin::rows_bucket(p.M)) {
    case 1: launch_pro<PRO, 1>(p, stream); break;
    case 2: launch_pro<PRO, 2>(p, stream); break;
    case 4: launch_pro<PRO, 4>(p, stream); break;
    default: launch_pro<PRO, 8>(p, stream); break;
  }
}

}  // namespace

hipError_t launch_linear(const LinearParams& p, hipStream_t stream) {
  if (p.M == 0 || p.N == 0) return hipSuccess;
  if (p.prologue == kProRmsNorm)
    launch_rows<kProRmsNorm>(p, stream);
  else if (p.prologue == kProSwiglu)
    launch_rows<kProSwiglu>(p, stream);
  else
    launch_rows<kProNone>(p, stream);
  return hipGetLastError();
}

}  // namespace qf
