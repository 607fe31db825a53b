// Fixed device scratch for the allocation-free one-launch decode (qf_attn_decode_noalloc).
//
// The one-launch decode keeps the partial states of every (shard, chunk) slot and one arrival
// counter per (request, KV head) in device memory beyond its inputs and outputs.  For callers that
// cannot allocate (graph capture, serving loops, harnesses that forbid hipMalloc) that memory is
// this file-scope array: every GPU the library runs on holds its own copy for the life of the
// process.  Host code never passes the array's name to a kernel (on the host it is only a stand-in
// for the symbol); the device address of each GPU's copy is looked up once per device with
// hipGetSymbolAddress and kept, and only that address is used.
#include <atomic>
#include <mutex>

#include "qf_internal.h"
#include "qfattn.h"

static_assert(QF_NOALLOC_SCRATCH_BYTES == qf::kNoallocScratchBytes, "scratch size of the header");
static_assert(QF_NOALLOC_STATE_BYTES == qf::kNoallocStateBytes, "state bytes of the header");
static_assert(QF_NOALLOC_MAX_GROUPS * sizeof(int32_t) == qf::kNoallocCounterBytes,
              "counter count of the header");

static __device__ __align__(256) unsigned char scratch[qf::kNoallocScratchBytes];

namespace qf {
namespace {

constexpr int kMaxDevices = 64;
std::atomic<unsigned char*> g_scratch[kMaxDevices];
std::mutex g_setup;

__global__ void __launch_bounds__(256) zero_i32(int32_t* __restrict__ p, int32_t n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
}

}  // namespace

hipError_t noalloc_prepare(int32_t n_counters, hipStream_t stream, int32_t** counters,
                           void** states) {
  if (n_counters < 0 || (size_t)n_counters * sizeof(int32_t) > kNoallocCounterBytes)
    return hipErrorInvalidValue;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  unsigned char* base = g_scratch[dev].load(std::memory_order_acquire);
  if (!base) {
    // Set-up, once per device, with that device current: its copy's address.
    std::lock_guard<std::mutex> lock(g_setup);
    base = g_scratch[dev].load(std::memory_order_relaxed);
    if (!base) {
      void* p = nullptr;
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return e;
      if (!p) return hipErrorInvalidSymbol;
      base = static_cast<unsigned char*>(p);
      g_scratch[dev].store(base, std::memory_order_release);
    }
  }
  *counters = reinterpret_cast<int32_t*>(base);
  *states = base + kNoallocCounterBytes;
  // The counters must start at zero.  The decode leaves the entries it used at zero, but the
  // array keeps whatever the last call on this GPU left, so they are cleared on every call, with
  // a kernel (no memset node if the caller captures the call into a graph).
  if (n_counters > 0) {
    hipLaunchKernelGGL(zero_i32, dim3((n_counters + 255) / 256), dim3(256), 0, stream, *counters,
                       n_counters);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace qf
