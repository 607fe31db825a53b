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
// One workgroup per (row, head); its wavefronts take the entries round-robin, every lane owns 2
// of the 128 dims, and the wavefronts' sums meet in LDS (they share the same m, so no rescale).
//
// With the current token (CUR): the merged pair is the cache's (o_<j, lse_<j), and the current
// token is folded in as §2 and Appendix A state it: s_jj = scale * q_j . k_j,
// out = lerp(v_j, o_<j, sigma(lse_<j - s_jj)) with sigma(x) = 1 / (1 + exp(-x)), and
// lse = logaddexp(lse_<j, s_jj).  An empty cache gives sigma(-inf) = 0, i.e. out = v_j.
#include <math.h>

#include "qf_internal.h"

namespace qf {
namespace {

constexpr int D = kHeadDim;
constexpr int W = kMergeWaves;

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

// fp32 -> bf16, round to nearest even; NaN stays a (quiet) NaN.
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x0040u;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <bool BF16, bool CUR>
__global__ void __launch_bounds__(64 * W)
merge_kernel(const float* __restrict__ in_o, const float* __restrict__ in_lse,
             void* __restrict__ out_o, float* __restrict__ out_lse, int32_t entries,
             int32_t hq, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cur,
             const uint16_t* __restrict__ v_cur, int32_t hkv, float scale) {
  const int pair = blockIdx.x;
  const int r = pair / hq;
  const int h = pair % hq;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const float* lse = in_lse + (size_t)r * entries * hq + h;
  const float2* o = reinterpret_cast<const float2*>(in_o + ((size_t)r * entries * hq + h) * D) + lane;
  const size_t o_step = (size_t)hq * D / 2;  // float2 between entries

  // m and the NaN flag over all entries, 64 entries per pass.
  float M = -INFINITY;
  int nan = 0;
  for (int i0 = 0; i0 < entries; i0 += 64) {
    const int i = i0 + lane;
    const float x = (i < entries) ? lse[(size_t)i * hq] : -INFINITY;
    nan |= (x != x);
    M = fmaxf(M, x);
  }
  M = wave_max(M);
  nan = __any(nan);

  float2 acc = make_float2(0.0f, 0.0f);
  float L = 0.0f;
  if (!nan && M != -INFINITY) {
    // Groups of 4 entries per wavefront: the loads of a group are issued together; a group whose
    // entries are all empty is skipped (unused shard slots sit at the end of a row).
    for (int i0 = 4 * wave; i0 < entries; i0 += 4 * W) {
      float x[4];
      bool live = false;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        x[k] = (i0 + k < entries) ? lse[(size_t)(i0 + k) * hq] : -INFINITY;
        live |= (x[k] != -INFINITY);
      }
      if (!live) continue;
      float2 v[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] = (i0 + k < entries) ? o[(size_t)(i0 + k) * o_step] : make_float2(0.0f, 0.0f);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (x[k] != -INFINITY) {
          const float w = expf(x[k] - M);
          L += w;
          acc.x = fmaf(w, v[k].x, acc.x);
          acc.y = fmaf(w, v[k].y, acc.y);
        }
      }
    }
  }

  __shared__ float2 s_acc[W][64];
  __shared__ float s_L[W];
  s_acc[wave][lane] = acc;
  if (lane == 0) s_L[wave] = L;
  __syncthreads();
  if (wave != 0) return;

  float2 a = s_acc[0][lane];
  float Lt = s_L[0];
#pragma unroll
  for (int w = 1; w < W; ++w) {
    a.x += s_acc[w][lane].x;
    a.y += s_acc[w][lane].y;
    Lt += s_L[w];
  }
  float lse_out;
  const size_t out_idx = ((size_t)r * hq + h) * D / 2 + lane;  // float2 / bf16-pair index
  if (nan) {
    a = make_float2(NAN, NAN);
    lse_out = NAN;
  } else if (M == -INFINITY) {
    a = make_float2(0.0f, 0.0f);
    lse_out = -INFINITY;
  } else {
    a.x /= Lt;
    a.y /= Lt;
    lse_out = M + logf(Lt);
  }
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
  } else if (M != -INFINITY || nan) {
    reinterpret_cast<float2*>(out_o)[out_idx] = a;
  }
  if (out_lse && lane == 0) out_lse[(size_t)r * hq + h] = lse_out;
}

}  // namespace

hipError_t launch_merge(const MergeParams& p, bool to_bf16, hipStream_t stream) {
  const unsigned grid = (unsigned)p.rows * (unsigned)p.hq;
  if (grid == 0) return hipSuccess;
  if (p.q)
    hipLaunchKernelGGL((merge_kernel<true, true>), dim3(grid), dim3(64 * W), 0, stream, p.in_o,
                       p.in_lse, p.out_o, p.out_lse, p.entries, p.hq, p.q, p.k_cur, p.v_cur,
                       p.hkv, p.scale);
  else if (to_bf16)
    hipLaunchKernelGGL((merge_kernel<true, false>), dim3(grid), dim3(64 * W), 0, stream, p.in_o,
                       p.in_lse, p.out_o, p.out_lse, p.entries, p.hq, nullptr, nullptr, nullptr,
                       1, 0.0f);
  else
    hipLaunchKernelGGL((merge_kernel<false, false>), dim3(grid), dim3(64 * W), 0, stream, p.in_o,
                       p.in_lse, p.out_o, p.out_lse, p.entries, p.hq, nullptr, nullptr, nullptr,
                       1, 0.0f);
  return hipGetLastError();
}

}  // namespace qf
