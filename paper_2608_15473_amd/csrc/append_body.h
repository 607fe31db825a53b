// Device body of the paged cache append of the current token (Q-First, arXiv:2608.15473, §2: k_j
// and v_j follow the query as a cache write nothing waits on), shared by the append kernel
// (kv_append.hip) and the merge that folds the current token in and appends it (merge.hip).
//
// One workgroup per request b: n = ctx_lens[b] is the slot the current token takes; its page is
// block_table[b, n / P] and its row n % P.  Each thread copies bf16 pairs of the KV heads' keys and
// values (2 * Hkv * 128 values per request).  When asked, the context length is advanced by one
// after every thread of the workgroup has read it, so no read can see the new value.  A position
// past the table's capacity, or a page outside the pool, writes nothing and sets *status = 1.
// Every thread of the workgroup must call it (it has a workgroup barrier when advancing).
#pragma once

#include "qf_internal.h"

namespace qf {
namespace app {

__device__ __forceinline__ void append_request(
    uint16_t* __restrict__ k, uint16_t* __restrict__ v, const int32_t* __restrict__ block_table,
    int32_t* __restrict__ ctx_lens, const uint16_t* __restrict__ k_new,
    const uint16_t* __restrict__ v_new, int32_t* __restrict__ status, int32_t hkv,
    int32_t max_pages, int32_t num_pages, int32_t advance, int b) {
  constexpr int D = kHeadDim;
  constexpr int P = kPage;
  const int n = ctx_lens[b];
  bool ok = n >= 0 && n < max_pages * P;
  int page = 0;
  if (ok) {
    page = block_table ? block_table[(size_t)b * max_pages + n / P] : b * max_pages + n / P;
    ok = (unsigned)page < (unsigned)num_pages;
  }
  if (ok) {
    const size_t row = ((size_t)page * hkv) * P * D + (size_t)(n % P) * D;  // head 0's row
    for (int i = threadIdx.x; i < hkv * D / 2; i += blockDim.x) {
      const int g = i / (D / 2);
      const int e = i % (D / 2);
      const size_t dst = row + (size_t)g * P * D;
      const size_t src = ((size_t)b * hkv + g) * D;
      reinterpret_cast<uint32_t*>(k + dst)[e] = reinterpret_cast<const uint32_t*>(k_new + src)[e];
      reinterpret_cast<uint32_t*>(v + dst)[e] = reinterpret_cast<const uint32_t*>(v_new + src)[e];
    }
  } else if (status && threadIdx.x == 0) {
    *status = 1;
  }
  if (advance) {
    __syncthreads();  // every thread has read ctx_lens[b]
    if (threadIdx.x == 0 && ok) ctx_lens[b] = n + 1;
  }
}

}  // namespace app
}  // namespace qf
