// Read-bandwidth probe: the ceiling that a plain streaming read reaches on
// this part, reported beside the fraction of the nominal HBM peak.  Every
// lane reads 16-byte words in a grid-stride loop, four independent loads in
// flight per iteration; the words are folded into one value per lane that
// is written only if it matches a constant no input is expected to produce,
// so the loads stay live without a write stream.
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
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    acc += (a.x ^ b.y) + (c.z ^ d.w) + (a.w ^ b.x) + (c.y ^ d.z);
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
  const int grid = 256 * 16;  // 16 workgroups of 256 threads per CU
  hipLaunchKernelGGL(k_read_probe, dim3(grid), dim3(kProbeThreads), 0, s, static_cast<const uint4*>(src), n16, sink);
  return hipGetLastError();
}

}  // namespace bgtq
