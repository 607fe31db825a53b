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
// One workgroup per (row, head); its wavefronts take the entries in groups of 16, every lane owns
// 2 of the 128 dims, and the wavefronts' sums meet in LDS.  The body is shared by the merge
// kernels and by the sweep's last workgroup of a (request, KV head) when the two are fused.
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

// Row r (request, or request x shard for a chunk merge), query head h of the partial states
// in_o [rows, entries, hq, D], in_lse [rows, entries, hq]: merged into out_o / out_lse, then (CUR)
// the current token folded in.  Called by every thread of a workgroup of W wavefronts.
// COHERENT: the partial states were written by other workgroups of the same launch (with
// device-scope stores), so they are read with device-scope loads, which bypass the XCD's
// non-coherent L2; the log-partitions would otherwise get scalar loads (a uniform address), whose
// cache would not see those writes either.
template <bool BF16, bool CUR, int W, bool COHERENT = false>
__device__ __forceinline__ void merge_row(
    const float* __restrict__ in_o, const float* __restrict__ in_lse, void* __restrict__ out_o,
    float* __restrict__ out_lse, int32_t entries, int32_t hq, const int r, const int h,
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cur,
    const uint16_t* __restrict__ v_cur, int32_t hkv, float scale) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const float* lse = in_lse + (size_t)r * entries * hq + h;
  const float2* o = reinterpret_cast<const float2*>(in_o + ((size_t)r * entries * hq + h) * D) + lane;
  const size_t o_step = (size_t)hq * D / 2;  // float2 between entries

  // Wavefront w takes entries [K w, K w + K) of every K W: its K log-partitions, then the O rows
  // of the live ones among them, all loaded before any is used.  Each wavefront keeps its own
  // running maximum m_w (rescaling its sums when a later group raises it), and the wavefronts
  // meet in LDS, where every sum is rescaled by exp(m_w - m).  Empty entries are selected out.
  // (Loading every O row together with the log-partitions, one round trip instead of two, was
  // measured no faster on MI355X, also where every entry is live.)
  constexpr int K = 16;
  float m_w = -INFINITY;
  float L = 0.0f;
  float2 acc = make_float2(0.0f, 0.0f);
  bool nan = false;
  for (int i0 = K * wave; i0 < entries; i0 += K * W) {
    float x[K];
    float2 v[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const bool in = i0 + k < entries;
      if (COHERENT)
        x[k] = in ? __hip_atomic_load(&lse[(size_t)(i0 + k) * hq], __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT)
                  : -INFINITY;
      else
        x[k] = in ? lse[(size_t)(i0 + k) * hq] : -INFINITY;
    }
    // O only where the slot holds positions: most slots of a ragged batch are empty, and their
    // O (never written) is not worth a read.
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const bool live = x[k] != -INFINITY;
      if (COHERENT) {
        const float* of = reinterpret_cast<const float*>(o + (size_t)(i0 + k) * o_step);
        v[k] = live ? make_float2(__hip_atomic_load(of, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT),
                                  __hip_atomic_load(of + 1, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT))
                    : make_float2(0.0f, 0.0f);
      } else {
        v[k] = live ? o[(size_t)(i0 + k) * o_step] : make_float2(0.0f, 0.0f);
      }
    }
    float mc = m_w;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      nan |= (x[k] != x[k]);
      mc = fmaxf(mc, x[k]);
    }
    if (mc == -INFINITY) continue;  // nothing live so far
    const float f = (m_w == -INFINITY) ? 0.0f : expf(m_w - mc);
    L *= f;
    acc.x *= f;
    acc.y *= f;
    m_w = mc;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const float w = (x[k] == -INFINITY) ? 0.0f : expf(x[k] - m_w);
      L += w;
      acc.x = (w == 0.0f) ? acc.x : fmaf(w, v[k].x, acc.x);
      acc.y = (w == 0.0f) ? acc.y : fmaf(w, v[k].y, acc.y);
    }
  }

  __shared__ float2 s_acc[W][64];
  __shared__ float s_L[W];
  __shared__ float s_m[W];
  __shared__ int s_nan[W];
  s_acc[wave][lane] = acc;
  if (lane == 0) {
    s_L[wave] = L;
    s_m[wave] = m_w;
    s_nan[wave] = nan;
  }
  __syncthreads();
  if (wave == 0) {
  float M = s_m[0];
  bool any_nan = s_nan[0];
#pragma unroll
  for (int w = 1; w < W; ++w) {
    M = fmaxf(M, s_m[w]);
    any_nan |= s_nan[w];
  }
  float2 a = make_float2(0.0f, 0.0f);
  float Lt = 0.0f;
#pragma unroll
  for (int w = 0; w < W; ++w) {
    const float f = (s_m[w] == -INFINITY) ? 0.0f : expf(s_m[w] - M);
    a.x = fmaf(f, s_acc[w][lane].x, a.x);
    a.y = fmaf(f, s_acc[w][lane].y, a.y);
    Lt = fmaf(f, s_L[w], Lt);
  }
  float lse_out;
  const size_t out_idx = ((size_t)r * hq + h) * D / 2 + lane;  // float2 / bf16-pair index
  if (any_nan) {
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
  } else if (M != -INFINITY || any_nan) {
    reinterpret_cast<float2*>(out_o)[out_idx] = a;
  }
  if (out_lse && lane == 0) out_lse[(size_t)r * hq + h] = lse_out;
  }
  __syncthreads();  // the LDS may be reused by a next call in the same workgroup
}

}  // namespace mrg
}  // namespace qf
