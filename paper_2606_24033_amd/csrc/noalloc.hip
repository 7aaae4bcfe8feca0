// Workspace of the decode entry point that allocates nothing
// (blockgtq_decode_attn_noalloc): the split counters and partials of
// blockgtq_decode_attn in a file-scope device array, one copy per GPU,
// held until the process ends.  Its address on the current device is taken
// once per device with hipGetSymbolAddress (the array's name in host code is
// only a host-side handle, never a device address).  Calls that overlap in
// time on one GPU share the array and race.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "blockgtq.h"
#include "kernels.h"

namespace bgtq {
namespace {

static __device__ __align__(256) uint8_t scratch[BGTQ_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

__global__ void k_clear_counters(int32_t* __restrict__ c, int n) {
  const int i = static_cast<int>(blockIdx.x * blockDim.x + threadIdx.x);
  if (i < n) c[i] = 0;
}

}  // namespace

hipError_t noalloc_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (p == nullptr) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));  // the current device's copy
      if (e != hipSuccess) return e;
      if (p == nullptr) return hipErrorInvalidSymbol;
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return hipSuccess;
}

hipError_t launch_clear_counters(int32_t* counters, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_clear_counters, dim3((n + 255) / 256), dim3(256), 0, s, counters, n);
  return hipGetLastError();
}

}  // namespace bgtq
