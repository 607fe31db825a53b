// The dense parts of a decoder block around the attention (Q-First, arXiv:2608.15473, §2): the
// projections W_q, W_k|W_v, W_o and the feed-forward M = W_down (silu(W_gate h) * W_up h), each
// fused with what feeds or follows it:
//   out = W . P(x) (+ residual),   P = identity | N(x) = x / sqrt(mean(x^2) + eps) * gain
//                                       | swiglu(x) = silu(x[:, :K]) * x[:, K:]
// The paper names N1, N2 only as normalisations and M as a feed-forward; the RMS form and the
// SwiGLU feed-forward are those of the Qwen3 blocks it converts.
//
// At decode a block sees a handful of rows (M <= 8), so each product is a weight stream: the
// kernel reads W once (N x K bf16, 16-byte loads), and the few input rows come from L1/L2.  One
// wavefront computes one output row n for every input row: its lanes stride K by 8 elements, each
// holding an fp32 partial per input row, reduced across the wavefront at the end.  The prologue is
// applied in registers; the residual add and the rounding to bf16 (nearest even) happen once, in
// the epilogue.
#pragma once

#include <math.h>

#include "qf_internal.h"

namespace qf {
namespace lin {

constexpr int kThreads = 256;           // 4 wavefronts = 4 output rows per workgroup
constexpr int kRowsPerBlock = kThreads / 64;

__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x0040u;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ void unpack8(uint4 v, float* f) {
  f[0] = lo(v.x); f[1] = hi(v.x); f[2] = lo(v.y); f[3] = hi(v.y);
  f[4] = lo(v.z); f[5] = hi(v.z); f[6] = lo(v.w); f[7] = hi(v.w);
}

__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

// Output rows of out = W . P(x) (+ residual): wavefront w of index bid takes rows
// (4 bid + w) R .. (4 bid + w) R + R - 1.
// PRO: kProNone, kProRmsNorm, kProSwiglu.  MB: input rows provided for (M <= MB).
// U: 512-element chunks of K each wavefront loads per group before using any; R: output rows per
// wavefront, all fed by the same input chunks (loaded and transformed once).  Neither changes the
// arithmetic: every lane accumulates each row's chunks in the same order for any U and R.
// GLU: the rows of W alternate gate and up (row 2i = gate i, 2i + 1 = up i; R even), and the
// output is the feed-forward's activation out[m, i] = silu(y[m, 2i]) * y[m, 2i + 1] (N / 2
// columns), computed once per element instead of in every row of the product that consumes it.
template <int PRO, int MB, int U, int R, bool GLU = false>
__device__ __forceinline__ void linear_rows(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
    const uint16_t* __restrict__ gain, const uint16_t* __restrict__ residual,
    uint16_t* __restrict__ out_a, uint16_t* __restrict__ out_b, int32_t M, int32_t N, int32_t K,
    int32_t n_split, float eps, const unsigned bid) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int x_stride = (PRO == kProSwiglu) ? 2 * K : K;

  const int n0 = ((int)bid * kRowsPerBlock + wave) * R;
  if (n0 >= N) return;
  const int vecs = K / 8;                 // 16-byte vectors per row
  // Buffer resources bound each row: a load past the end returns 0 with no branch, so every
  // load of a group is issued unconditionally (rows past N get an empty range).  The weight stream
  // is read once (non-temporal); the input rows and gains are read by every workgroup (default).
  __amdgpu_buffer_rsrc_t rw[R];
#pragma unroll
  for (int r = 0; r < R; ++r)
    rw[r] = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(w + (size_t)(n0 + r < N ? n0 + r : n0) * K), (short)0,
        n0 + r < N ? K * 2 : 0, 0x00020000);
  const __amdgpu_buffer_rsrc_t rg = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(gain ? gain : w), (short)0, PRO == kProRmsNorm ? K * 2 : 0, 0x00020000);
  __amdgpu_buffer_rsrc_t rx[MB];
#pragma unroll
  for (int m = 0; m < MB; ++m)
    rx[m] = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(x + (size_t)(m < M ? m : 0) * x_stride), (short)0,
        m < M ? x_stride * 2 : 0, 0x00020000);
  // With the RMS prologue the normalisation factor r_m is a scalar per input row, so the wavefront
  // accumulates sum_k W[n,k] x[m,k] g[k] and sum_k x[m,k]^2 over the same chunks and applies
  // r_m = 1 / sqrt(mean x^2 + eps) once at the end: no separate pass over x, no barrier.
  float acc[R][MB], ss[MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) {
    ss[m] = 0.0f;
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r][m] = 0.0f;
  }

  // Per group of U chunks every load the group needs (weights, inputs, gains) is issued before
  // any is used: wait counts are in order, so one wait then covers the whole group.
  for (int c0 = 0; c0 < vecs; c0 += 64 * U) {
    uint4 wv[U][R], xv[U][MB], uv[PRO == kProSwiglu ? U : 1][PRO == kProSwiglu ? MB : 1],
        gv[PRO == kProRmsNorm ? U : 1];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int off = (c0 + u * 64) * 16;                 // uniform byte offset of the chunk
      const int vo = (c0 + u * 64 + lane < vecs) ? lane * 16 : K * 4;   // past the end: 0
#pragma unroll
      for (int r = 0; r < R; ++r)
        wv[u][r] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rw[r], vo, off, 2));
      if (PRO == kProRmsNorm)
        gv[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rg, vo, off, 0));
#pragma unroll
      for (int m = 0; m < MB; ++m) {
        xv[u][m] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rx[m], vo, off, 0));
        if (PRO == kProSwiglu)
          uv[u][m] = __builtin_bit_cast(
              uint4, __builtin_amdgcn_raw_buffer_load_b128(rx[m], vo, off + K * 2, 0));
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float g[8];
      if (PRO == kProRmsNorm) unpack8(gv[u], g);
#pragma unroll
      for (int m = 0; m < MB; ++m) {
        float xf[8];
        unpack8(xv[u][m], xf);
        if (PRO == kProRmsNorm) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            ss[m] = fmaf(xf[j], xf[j], ss[m]);
            xf[j] *= g[j];
          }
        } else if (PRO == kProSwiglu) {
          float up[8];
          unpack8(uv[u][m], up);
#pragma unroll
          for (int j = 0; j < 8; ++j) xf[j] = silu(xf[j]) * up[j];
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
          float wf[8];
          unpack8(wv[u][r], wf);
#pragma unroll
          for (int j = 0; j < 8; ++j) acc[r][m] = fmaf(wf[j], xf[j], acc[r][m]);
        }
      }
    }
  }

#pragma unroll
  for (int m = 0; m < MB; ++m) {
    float scale = 1.0f;
    if (PRO == kProRmsNorm) {
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) ss[m] += __shfl_xor(ss[m], o);
      scale = 1.0f / sqrtf(ss[m] / (float)K + eps);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) acc[r][m] += __shfl_xor(acc[r][m], o);
      if (PRO == kProRmsNorm) acc[r][m] *= scale;
    }
  }
  if (GLU) {
    static_assert(!GLU || R % 2 == 0, "gate and up rows come in pairs");
    if (lane < M) {
#pragma unroll
      for (int r = 0; r < R; r += 2) {
        if (n0 + r + 1 >= N) break;
        float g = 0.0f, v = 0.0f;
#pragma unroll
        for (int m = 0; m < MB; ++m)
          if (m == lane) {
            g = acc[r][m];
            v = acc[r + 1][m];
          }
        out_a[(size_t)lane * (N / 2) + (n0 + r) / 2] = (uint16_t)bf16_rne(silu(g) * v);
      }
    }
    return;
  }
  if (lane < M) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int n = n0 + r;
      if (n >= N) break;
      float y = 0.0f;
#pragma unroll
      for (int m = 0; m < MB; ++m)
        if (m == lane) y = acc[r][m];
      if (residual) y += lo(residual[(size_t)lane * N + n]);
      const uint16_t b = (uint16_t)bf16_rne(y);
      if (n < n_split)
        out_a[(size_t)lane * n_split + n] = b;
      else
        out_b[(size_t)lane * (N - n_split) + (n - n_split)] = b;
    }
  }
}

// Workgroups a product of N output rows needs at R rows per wavefront.
inline int linear_blocks(int N, int R) { return (N + kRowsPerBlock * R - 1) / (kRowsPerBlock * R); }

// R for the shared launch with the sweep, where the product's workgroups run at the sweep's
// occupancy: more rows per wavefront keep enough weight bytes in flight.
constexpr int beside_rows(int MB) { return MB <= 2 ? 4 : MB <= 4 ? 2 : 1; }
constexpr int beside_rows_glu(int MB) { return MB <= 2 ? 4 : 2; }

// U for a row length K: enough chunks to cover K in one group where registers allow (at most 8
// loads of weights plus 8 of inputs per lane).
inline int pick_unroll(int M, int K) {
  const int cap = (M <= 1) ? 8 : (M <= 2) ? 4 : (M <= 4) ? 2 : 1;
  const int need = (K / 8 + 63) / 64;
  int u = 1;
  while (u < cap && u < need) u *= 2;
  return u;
}

inline int rows_bucket(int M) { return (M <= 1) ? 1 : (M <= 2) ? 2 : (M <= 4) ? 4 : 8; }

}  // namespace lin
}  // namespace qf
