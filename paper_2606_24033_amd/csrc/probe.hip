// Read-bandwidth probe: the ceiling that a plain streaming read reaches on
// this part, reported beside the fraction of the nominal HBM peak.  Every
// lane reads 16-byte words in a grid-stride loop, four independent
// nontemporal loads in flight per iteration, 32 workgroups of 256 lanes per
// CU (the fastest of the read patterns swept on MI355X: 6.4-6.6 TB/s); the
// words are folded into one value per lane that is written only if it
// matches a constant no input is expected to produce, so the loads stay live
// without a write stream.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace bgtq {
namespace {

constexpr int kProbeThreads = 256;

__global__ __launch_bounds__(kProbeThreads) void k_read_probe(const uint4* __restrict__ src, size_t n16,
                                                              uint32_t* __restrict__ sink) {
  const size_t stride = static_cast<size_t>(gridDim.x) * kProbeThreads;
  size_t i = static_cast<size_t>(blockIdx.x) * kProbeThreads + threadIdx.x;
  uint32_t acc = 0;
  typedef unsigned int u4v __attribute__((ext_vector_type(4)));
  const u4v* s4 = reinterpret_cast<const u4v*>(src);
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u4v a = __builtin_nontemporal_load(s4 + i), b = __builtin_nontemporal_load(s4 + i + stride);
    const u4v c = __builtin_nontemporal_load(s4 + i + 2 * stride), d = __builtin_nontemporal_load(s4 + i + 3 * stride);
    acc += (a[0] ^ b[1]) + (c[2] ^ d[3]) + (a[3] ^ b[0]) + (c[1] ^ d[2]);
  }
  for (; i < n16; i += stride) {
    const uint4 a = src[i];
    acc += a.x ^ a.w;
  }
  if (acc == 0x9E3779B9u) sink[0] = acc;
}

}  // namespace

hipError_t launch_read_probe(const void* src, size_t bytes, uint32_t* sink, hipStream_t s) {
  const size_t n16 = bytes / 16;
  const int grid = 256 * 32;  // 32 workgroups of 256 threads per CU
  hipLaunchKernelGGL(k_read_probe, dim3(grid), dim3(kProbeThreads), 0, s, static_cast<const uint4*>(src), n16, sink);
  return hipGetLastError();
}

}  // namespace bgtq
