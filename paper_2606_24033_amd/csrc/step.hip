// Decode step from pre-RoPE inputs: RoPE applied on the device (Sec. 2.1 and
// Sec. 2.3: block i of a vector at position t is rotated by the angle
// t * theta_i, theta_i = base^(-2i/d_h), block i = dims (i, i + d_h/2)), then
// the append and the packed decode of every layer.  The angles are formed and
// reduced in fp64, so a position of 10^6 loses nothing to fp32 angle error.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "layout.h"

namespace bgtq {
namespace {

__device__ __forceinline__ float ld_in(const void* p, size_t i, int dtype) {  // BGTQ_BF16 = 1
  if (dtype == 1) return __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(p)[i]) << 16);
  return reinterpret_cast<const float*>(p)[i];
}

// grid (n_lc * batch, Hq + n_kv), 64 threads (thread = RoPE block i).  Head
// slots below Hq rotate a query head; the others rotate a key head and copy
// its value row.  Outputs are fp32: q [n_lc][batch][Hq][128], k and v
// [n_lc][batch][1][n_kv][128]; ctx[b] = pos[b] + 1.
__global__ __launch_bounds__(64) void k_rope_step(Dims d, double base, const void* __restrict__ q,
                                                  const void* __restrict__ k, const void* __restrict__ v,
                                                  const int32_t* __restrict__ pos, float* __restrict__ qo,
                                                  float* __restrict__ ko, float* __restrict__ vo,
                                                  int32_t* __restrict__ ctx) {
  const int lz = blockIdx.x, slot = blockIdx.y, i = threadIdx.x;
  const int seq = lz % d.batch;
  const int hq = d.n_kv * d.group;
  const int p = pos[seq];
  if (lz < d.batch && slot == 0 && i == 0) ctx[seq] = p + 1;
  // angle p * theta_i in fp64, reduced into [-pi, pi] before sin / cos
  const double theta = pow(base, -2.0 * i / kHeadDim);
  double phi = static_cast<double>(p) * theta;
  phi -= 6.283185307179586 * rint(phi * 0.15915494309189535);
  double sn, cs;
  sincos(phi, &sn, &cs);
  size_t off;
  const void* src;
  float* dst;
  if (slot < hq) {
    off = (static_cast<size_t>(lz) * hq + slot) * kHeadDim;
    src = q;
    dst = qo;
  } else {
    off = (static_cast<size_t>(lz) * d.n_kv + (slot - hq)) * kHeadDim;
    src = k;
    dst = ko;
    vo[off + i] = ld_in(v, off + i, d.in_dtype);
    vo[off + i + 64] = ld_in(v, off + i + 64, d.in_dtype);
  }
  const double x0 = ld_in(src, off + i, d.in_dtype), x1 = ld_in(src, off + i + 64, d.in_dtype);
  dst[off + i] = static_cast<float>(x0 * cs - x1 * sn);
  dst[off + i + 64] = static_cast<float>(x0 * sn + x1 * cs);
}

}  // namespace

hipError_t launch_rope_step(const Dims& d, double base, const void* q, const void* k, const void* v,
                            const int32_t* pos, float* qo, float* ko, float* vo, int32_t* ctx, hipStream_t s) {
  dim3 grid(d.n_lc * d.batch, d.n_kv * d.group + d.n_kv);
  hipLaunchKernelGGL(k_rope_step, grid, dim3(64), 0, s, d, base, q, k, v, pos, qo, ko, vo, ctx);
  return hipGetLastError();
}

}  // namespace bgtq
