// HIP kernels of the Block-GTQ packed-cache path for gfx950 (MI355X).
//
//  k_append_rows   : TQ-MSE encode (Sec. 2.2) of a few appended K rows per
//                    same-rate group (end of Sec. 3.2) and of their V rows,
//                    dense b-bit pack (decode steps).
//  (long appends run on fp32 MFMAs in quantize.hip; the packed-cache decode
//  and the fp16 comparator live in decode_impl.h)
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "layout.h"

namespace bgtq {

namespace {

constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ float ld_in(const void* p, size_t i, int dtype) {
  if (dtype == 1) {
    uint32_t u = reinterpret_cast<const uint16_t*>(p)[i];
    return __uint_as_float(u << 16);
  }
  return reinterpret_cast<const float*>(p)[i];
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Number of thresholds t with t <= z (2^b - 1 sorted thresholds).
__device__ __forceinline__ int scalar_code(const float* thr, int b, float z) {
  int idx = 0;
  for (int step = 1 << (b - 1); step > 0; step >>= 1)
    if (thr[idx + step - 1] <= z) idx += step;
  return idx;
}

// ---------------------------------------------------------------------------
// Decode-step append: n_new <= kRowAppend rows per (KV head, sequence[,
// layer]), one 1024-thread workgroup each.  The encode of Sec. 2.2 per
// same-rate group, and of the value row, arranged for latency:
// every global read is issued in one round, each thread's 32 rotation
// coefficients in flight together and used for all the rows.  Threads
// [0, 512): key stream position p = tid % 128 and summation quarter tid / 128
// (terms 32 qq .. 32 qq + 31 of its group); threads [512, 1024): value
// coordinate j and quarter.  The quarters are added in order, 0 to 3.
// ---------------------------------------------------------------------------
constexpr int kRowAppend = 4;

template <bool BF16>
__global__ __launch_bounds__(1024) void k_append_rows(Dims d, const uint8_t* __restrict__ blob,
                                                      const void* __restrict__ kin,
                                                      const void* __restrict__ vin, int n_new,
                                                      const int32_t* __restrict__ wpos, CachePtrs c) {
  __shared__ float xk[kRowAppend][kHeadDim];
  __shared__ float xv[kRowAppend][kHeadDim];
  __shared__ float pk[kRowAppend][4][kHeadDim];  // quarter sums of the rotated key positions
  __shared__ float pv[kRowAppend][4][kHeadDim];  // and of the rotated value coordinates
  __shared__ float nrm[kRowAppend][kMaxGroups + 1];
  __shared__ float thr[kThresholdEntries];
  __shared__ uint32_t dimw[kHeadDim / 4];        // RowMeta::dim
  __shared__ uint16_t boff[kHeadDim];            // RowMeta::bitoff
  __shared__ float xs[kRowAppend][kHeadDim];     // key rows in stream order: xs[s][p] = xk[s][dim(p)]
  __shared__ uint32_t kwd[kRowAppend][kMaxKWords];  // packed key rows
  __shared__ uint8_t cv[kRowAppend][kHeadDim];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.x, lz = blockIdx.y;
  const int layer = d.layer >= 0 ? d.layer : lz / d.batch;
  const int seq = lz % d.batch;
  const int cap = d.capacity;
  const RowMeta* M = reinterpret_cast<const RowMeta*>(blob + kOffRows) + (layer * d.n_kv + head);
  const float* rotkt = reinterpret_cast<const float*>(blob + kOffRotKT);
  const float* rotvt = reinterpret_cast<const float*>(blob + kOffRotVT);
  const float* gthr = reinterpret_cast<const float*>(blob + kOffThr);
  const size_t row = (static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + head;

  // group table (wave-uniform); the group of key position p is the last one
  // that starts at or before p
  const int ng = M->n_groups;
  int gdim[kMaxGroups], gpos[kMaxGroups], gbits[kMaxGroups];
#pragma unroll
  for (int g = 0; g < kMaxGroups; ++g) {  // whole arrays read, entries past n_g replaced
    const int a = M->g_dim[g], b = M->g_pos[g], w = M->g_bits[g];
    gdim[g] = g < ng ? a : 0;
    gpos[g] = g < ng ? b : kHeadDim;
    gbits[g] = g < ng ? w : 1;
  }
  // ---- one round of global reads
  const int p = tid & 127, qq = (tid >> 7) & 3;
  // the group of key position p (select chains with constant indices keep the
  // group table in registers)
  int dg = gdim[0], p0 = gpos[0], bk = gbits[0], gk = 0;
#pragma unroll
  for (int h = 1; h < kMaxGroups; ++h)
    if (p >= gpos[h]) {
      dg = gdim[h];
      p0 = gpos[h];
      bk = gbits[h];
      gk = h;
    }
  // key threads: column j = p - p0 of Pi_dg transposed (rows past d_g re-read
  // the last one and are never used); value threads: column p of Pi_V^T.
  // One straight-line block, so that all 32 loads are in flight together.
  const bool kside = tid < 512;
  const float* rsrc = kside ? rotkt + rotk_index(dg) + (p - p0) : rotvt + p;
  const int rstride = kside ? dg : kHeadDim, rlast = kside ? dg - 1 : kHeadDim - 1;
  float rc[32];
#pragma unroll
  for (int u = 0; u < 32; ++u) rc[u] = rsrc[min(32 * qq + u, rlast) * rstride];
  // the other reads take clamped indices (in bounds, surplus values unused)
  // so that they need no branch either
  const size_t xoff =
      ((static_cast<size_t>(lz) * n_new + min(tid >> 7, n_new - 1)) * d.n_kv + head) * kHeadDim + p;
  float xkv, xvv;
  if constexpr (BF16) {
    xkv = __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(kin)[xoff]) << 16);
    xvv = __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(vin)[xoff]) << 16);
  } else {
    xkv = reinterpret_cast<const float*>(kin)[xoff];
    xvv = reinterpret_cast<const float*>(vin)[xoff];
  }
  const float tv = gthr[min(tid, kThresholdEntries - 1)];
  const uint32_t mw = reinterpret_cast<const uint32_t*>(M->dim)[tid & (kHeadDim / 4 - 1)];
  const uint32_t bw = reinterpret_cast<const uint32_t*>(M->bitoff)[tid & (kHeadDim / 2 - 1)];
  // the value words of the first row (value thread j = tid - 512 < 128), read
  // here so that its read-modify-write costs no extra round trip
  const int wp = wpos[seq];
  const int bv = d.v_bits;
  const int vj = (tid - 512) & 127;
  const int wp0 = min(max(wp, 0), cap - 1);
  const int vbit0 = (wp0 % kTile) * bv, vw0 = vbit0 >> 5;
  uint32_t* const vrow0 = c.v_codes + ((row * (cap / kTile) + wp0 / kTile) * kHeadDim + vj) * static_cast<size_t>(bv);
  const uint32_t v0lo = vrow0[vw0], v0hi = vrow0[min(vw0 + 1, bv - 1)];
  if (wp < 0 || wp >= cap) return;
  const int nt = min(n_new, cap - wp);  // rows that fit (the host rejects overflow)
  if (tid < nt * kHeadDim) {
    xk[tid >> 7][p] = xkv;
    xv[tid >> 7][p] = xvv;
  }
  if (tid < kThresholdEntries) thr[tid] = tv;
  if (tid < kHeadDim / 4) dimw[tid] = mw;
  if (tid < kHeadDim / 2) reinterpret_cast<uint32_t*>(boff)[tid] = bw;
  if (tid < kRowAppend * kMaxKWords) kwd[tid / kMaxKWords][tid % kMaxKWords] = 0u;
  __syncthreads();
  const uint8_t* dimp = reinterpret_cast<const uint8_t*>(dimw);
  if (tid < nt * kHeadDim) xs[tid >> 7][p] = xk[tid >> 7][dimp[p]];
  __syncthreads();

  // ---- group and value-row norms (one wave per (row, group)), quarter sums
  for (int item = wave; item < nt * (kMaxGroups + 1); item += 16) {
    const int s = item / (kMaxGroups + 1), g = item - s * (kMaxGroups + 1);
    if (g < ng) {
      // the group's extent by a select chain (a runtime index would put the
      // group table in scratch memory)
      int gd = gdim[0], gp = gpos[0];
#pragma unroll
      for (int h = 1; h < kMaxGroups; ++h)
        if (g == h) {
          gd = gdim[h];
          gp = gpos[h];
        }
      float ss = 0.f;
      for (int i = lane; i < gd; i += 64) {
        const float x = xs[s][gp + i];
        ss = fmaf(x, x, ss);
      }
      ss = wave_sum(ss);
      if (lane == 0) nrm[s][g] = sqrtf(ss);
    } else if (g == kMaxGroups) {
      float ss = 0.f;
      for (int i = lane; i < kHeadDim; i += 64) ss = fmaf(xv[s][i], xv[s][i], ss);
      ss = wave_sum(ss);
      if (lane == 0) nrm[s][kMaxGroups] = sqrtf(ss);
    }
  }
  for (int s = 0; s < nt; ++s) {
    float a = 0.f;
    if (kside) {
#pragma unroll
      for (int u = 0; u < 32; ++u)
        if (32 * qq + u < dg) a = fmaf(rc[u], xs[s][p0 + 32 * qq + u], a);
      pk[s][qq][p] = a;
    } else {
#pragma unroll
      for (int u = 0; u < 32; ++u) a = fmaf(rc[u], xv[s][32 * qq + u], a);
      pv[s][qq][p] = a;
    }
  }
  __syncthreads();

  // ---- codes (nearest centroid = count of thresholds <= z) and radii
  if (tid < kHeadDim) {
    for (int s = 0; s < nt; ++s) {
      const float z = (pk[s][0][p] + pk[s][1][p]) + (pk[s][2][p] + pk[s][3][p]);
      const float n = nrm[s][gk];
      const float scale = n > 0.f ? sqrtf(static_cast<float>(dg)) / n : 0.f;
      // the code's bits [boff, boff + b) go into the packed row (LDS or)
      const uint32_t code = static_cast<uint32_t>(scalar_code(thr + thr_index(bk), bk, z * scale));
      const int bo = boff[p], w = bo >> 5, sh = bo & 31;
      atomicOr(&kwd[s][w], code << sh);
      if (sh + bk > 32) atomicOr(&kwd[s][w + 1], code >> (32 - sh));
      if (p == p0)
        c.k_norms[row * kMaxGroups * cap + static_cast<size_t>(wp + s) * ((ng + 1) & ~1) + gk] =
            __half_as_ushort(__float2half_rn(n));
    }
  } else if (tid < 2 * kHeadDim) {
    const int bv = d.v_bits;
    for (int s = 0; s < nt; ++s) {
      const float z = (pv[s][0][p] + pv[s][1][p]) + (pv[s][2][p] + pv[s][3][p]);
      const float n = nrm[s][kMaxGroups];
      const float scale = n > 0.f ? sqrtf(static_cast<float>(kHeadDim)) / n : 0.f;
      cv[s][p] = static_cast<uint8_t>(scalar_code(thr + thr_index(bv), bv, z * scale));
      if (p == 0) c.v_norms[row * cap + wp + s] = __half_as_ushort(__float2half_rn(n));
    }
  }
  __syncthreads();

  // ---- pack: whole key words; the value slots of the rows inside their tiles
  const int kw = d.k_words;
  if (tid < nt * kw) {
    const int s = tid / kw, w = tid - s * kw;
    c.k_codes[(row * cap + wp + s) * kw + w] = kwd[s][w];
  } else if (tid >= 512 && tid < 512 + kHeadDim) {
    const int j = vj;
    const uint32_t mask = (1u << bv) - 1u;
    for (int s = 0; s < nt; ++s) {
      const int t = wp + s, slot = t % kTile, bit = slot * bv, w = bit >> 5, sh = bit & 31;
      uint32_t* vw = c.v_codes + ((row * (cap / kTile) + t / kTile) * kHeadDim + j) * static_cast<size_t>(bv);
      const uint32_t code = cv[s][j];
      // row 0 starts from the words read up front; later rows re-read (a row
      // may share a word with the previous one)
      const uint32_t lo = s == 0 ? v0lo : vw[w];
      vw[w] = (lo & ~(mask << sh)) | (code << sh);
      if (sh + bv > 32) {
        const int hi = sh + bv - 32;  // bits of the code in the next word
        const uint32_t up = s == 0 ? v0hi : vw[w + 1];
        vw[w + 1] = (up & ~((1u << hi) - 1u)) | (code >> (bv - hi));
      }
    }
  }
}

}  // namespace

hipError_t launch_quantize_append(const Dims& d, const void* layout, const void* k, const void* v,
                                  int n_new, const int32_t* write_pos, const CachePtrs& c,
                                  hipStream_t s) {
  if (n_new <= 0) return hipSuccess;
  if (n_new <= kRowAppend) {
    const auto kern = d.in_dtype == 1 ? k_append_rows<true> : k_append_rows<false>;
    hipLaunchKernelGGL(kern, dim3(d.n_kv, d.batch * d.n_lc), dim3(1024), 0, s, d,
                       static_cast<const uint8_t*>(layout), k, v, n_new, write_pos, c);
    return hipGetLastError();
  }
  return launch_quantize_prefill(d, layout, k, v, n_new, write_pos, c, s);
}

hipError_t launch_decode_packed(const Dims& d, const void* layout, const void* q,
                                const int32_t* ctx_len, const CachePtrs& c, float* out,
                                const DecodeWs& ws, hipStream_t s) {
  switch (d.v_bits) {
    case 1: return launch_split_bv1(d, layout, q, ctx_len, c, out, ws, s);
    case 2: return launch_split_bv2(d, layout, q, ctx_len, c, out, ws, s);
    case 3: return launch_split_bv3(d, layout, q, ctx_len, c, out, ws, s);
    case 4: return launch_split_bv4(d, layout, q, ctx_len, c, out, ws, s);
    case 5: return launch_split_bv5(d, layout, q, ctx_len, c, out, ws, s);
    case 6: return launch_split_bv6(d, layout, q, ctx_len, c, out, ws, s);
    case 7: return launch_split_bv7(d, layout, q, ctx_len, c, out, ws, s);
    default: return launch_split_bv8(d, layout, q, ctx_len, c, out, ws, s);
  }
}


}  // namespace bgtq
