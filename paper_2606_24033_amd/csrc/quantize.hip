// Prefill quantize + pack + append on fp32 MFMAs: the TQ-MSE encode of
// Sec. 2.2 applied to every same-rate group of a key row (end of Sec. 3.2)
// and to the value row, for the long appends of a prefill (Sec. 4, prefill
// paragraph).  Appends of a few rows (decode steps) use k_append_rows.
//
// Both encodes are dense 128 x 128 products per row on
// v_mfma_f32_16x16x4f32 (16 rows of a wave at a time), with the reduction
// index arranged so that a lane's 32 k-steps read 32 contiguous input dims
// (k-step s of lane l pairs with dim 32 (l / 16) + s): a lane loads its slice
// of a row with 16-byte loads and no gather.
//
// One launch (k_quant_rows) for both: its first workgroups encode keys, the
// others values.
//  keys   : Z = W X^T.  W (the layout's dense key rotation on the natural
//           dims, the gather into stream order folded in) is the A operand,
//           staged in LDS once per workgroup; the key rows are the B
//           operand.  A lane ends with four consecutive stream positions of
//           one row, i.e. one contiguous bit field of the packed row.  The
//           group radii come from the same kind of product, a 0/1 group
//           membership matrix times the squared inputs.
//  values : Z = X Pi_V^T.  The value rows are the A operand, Pi_V the B
//           operand.  A lane ends with one coordinate of four consecutive
//           rows, i.e. one contiguous bit field of a 32-row value tile.
// Codes: number of thresholds <= z (binary search over the fp32 midpoints of
// the fp16 centroids, LDS); rows and tiles are assembled in LDS with atomic
// ORs and written with whole-word stores.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "layout.h"

namespace bgtq {
namespace quant_detail {

typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kWaves = 16;
constexpr int kThreads = kWaves * 64;
constexpr int kSub = 16;                          // rows per wave sub-tile (one MFMA column block)
constexpr int kMatF4 = kMfmaMatFloats / 4;        // float4 entries of one MFMA-order matrix

struct LdsK {
  float4 wa[kMatF4];                          // the row's W, A operand order
  float4 ma[8 * 64];                          // group membership, A operand order ([s4][lane])
  uint32_t rw[kWaves][kSub][kMaxKWords];      // per wave: packed key rows
  float sc[kWaves][kSub][kMaxGroups];         // per wave: sqrt(d_g) / radius of each row and group
  float thr[kThresholdEntries];
  uint32_t pm[kHeadDim];                      // per stream position: bit offset | b << 10 | group << 14
  float gs[kMaxGroups];                       // sqrt(d_g)
  uint8_t gd[kHeadDim];                       // group ordinal of each input dim
};
struct LdsV {
  float4 rb[kMatF4];                          // Pi_V, B operand order
  uint32_t vt[kWaves][kHeadDim][8];           // per wave: words of one value tile
  float nv[kWaves][32];                       // per wave: the tile's value radii
  float thr[kThresholdEntries];
};
static_assert(sizeof(LdsK) <= 160 * 1024 && sizeof(LdsV) <= 160 * 1024, "LDS of one workgroup");

__device__ __forceinline__ void wave_sync() {
  // LDS operations of one wave complete in order; only the compiler must
  // keep them in program order
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Number of thresholds t <= z among the 2^b - 1 sorted thresholds at thr.
__device__ __forceinline__ uint32_t scalar_code(const float* thr, int b, float z) {
  int idx = 0;
  for (int step = 1 << (b - 1); step > 0; step >>= 1)
    if (thr[idx + step - 1] <= z) idx += step;
  return static_cast<uint32_t>(idx);
}

// Dims [32 kk, 32 kk + 32) of one input row (zeros when !valid); the row
// starts 16-byte aligned (the host checks the base pointer).
template <bool BF16>
__device__ __forceinline__ void load_slice(const void* src, size_t elem_off, bool valid, float (&x)[32]) {
  if (!valid) {
#pragma unroll
    for (int i = 0; i < 32; ++i) x[i] = 0.f;
    return;
  }
  if constexpr (BF16) {
    const uint4* p = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(src) + elem_off);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint4 v = p[q];
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[8 * q + 2 * e] = __uint_as_float(w[e] << 16);
        x[8 * q + 2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
      }
    }
  } else {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(src) + elem_off);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const float4 v = p[q];
      x[4 * q] = v.x;
      x[4 * q + 1] = v.y;
      x[4 * q + 2] = v.z;
      x[4 * q + 3] = v.w;
    }
  }
}

__device__ __forceinline__ float4_t mfma(float a, float b, float4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------- keys
// Workgroup bx of the key part: rows [bx R, bx R + R) of the call, R =
// kWaves kSub iters.
template <bool BF16>
__device__ __forceinline__ void quant_keys(LdsK& S, int bx, int iters, const Dims& d,
                                           const uint8_t* __restrict__ blob, const void* __restrict__ kin, int n_new,
                                           const int32_t* __restrict__ wpos, const CachePtrs& c) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.y, lz = blockIdx.z;
  const int layer = d.layer >= 0 ? d.layer : lz / d.batch;
  const int seq = lz % d.batch;
  const int cap = d.capacity;
  const int wp = wpos[seq];
  if (wp < 0 || wp >= cap) return;
  const int n_fit = min(n_new, cap - wp);  // rows that fit (the host rejects overflow)
  const int r_wg = bx * kWaves * kSub * iters;
  if (r_wg >= n_fit) return;
  const int n_rows_blob = d.n_layers * d.n_kv;
  const int ri = layer * d.n_kv + head;
  const RowMeta* M = reinterpret_cast<const RowMeta*>(blob + kOffRows) + ri;
  const float4* wsrc = reinterpret_cast<const float4*>(blob + layout_kdense_offset(n_rows_blob)) +
                       static_cast<size_t>(ri) * kMatF4;
  const float* gthr = reinterpret_cast<const float*>(blob + kOffThr);
  const int ng = M->n_groups;

  for (int i = tid; i < kMatF4; i += kThreads) S.wa[i] = wsrc[i];
  for (int i = tid; i < kWaves * kSub * kMaxKWords; i += kThreads) (&S.rw[0][0][0])[i] = 0u;
  for (int i = tid; i < kThresholdEntries; i += kThreads) S.thr[i] = gthr[i];
  if (tid < kHeadDim) {
    const int g = M->grp[tid];
    S.gd[M->dim[tid]] = static_cast<uint8_t>(g);
    S.pm[tid] = static_cast<uint32_t>(M->bitoff[tid]) | (static_cast<uint32_t>(M->width[tid]) << 10) |
                (static_cast<uint32_t>(g) << 14);
  }
  if (tid < kMaxGroups) S.gs[tid] = tid < ng ? sqrtf(static_cast<float>(M->g_dim[tid])) : 0.f;
  __syncthreads();
  for (int i = tid; i < 8 * 64; i += kThreads) {
    const int s4 = i >> 6, l = i & 63, g = l & 15, d0 = 32 * (l >> 4) + 4 * s4;
    S.ma[i] = make_float4(S.gd[d0] == g ? 1.f : 0.f, S.gd[d0 + 1] == g ? 1.f : 0.f, S.gd[d0 + 2] == g ? 1.f : 0.f,
                          S.gd[d0 + 3] == g ? 1.f : 0.f);
  }
  __syncthreads();

  const int tk = lane & 15, kk = lane >> 4;
  const int kw = d.k_words, nslot = (ng + 1) & ~1;
  const size_t row = (static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + head;
  for (int it = 0; it < iters; ++it) {
    const int r0 = r_wg + (it * kWaves + wave) * kSub;
    if (r0 >= n_fit) break;  // wave-uniform
    const int r = r0 + tk;
    const bool valid = r < n_fit;
    float x[32];
    load_slice<BF16>(kin, ((static_cast<size_t>(lz) * n_new + r) * d.n_kv + head) * kHeadDim + 32 * kk, valid, x);

    // group radii: R2[g][row] = sum_d [group(d) = g] x[row][d]^2
    float4_t n2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s4 = 0; s4 < 8; ++s4) {
      const float4 m = S.ma[s4 * 64 + lane];
      n2 = mfma(m.x, x[4 * s4] * x[4 * s4], n2);
      n2 = mfma(m.y, x[4 * s4 + 1] * x[4 * s4 + 1], n2);
      n2 = mfma(m.z, x[4 * s4 + 2] * x[4 * s4 + 2], n2);
      n2 = mfma(m.w, x[4 * s4 + 3] * x[4 * s4 + 3], n2);
    }
    // rotation: Z[p][row] = sum_d W[p][d] x[row][d], 8 tiles of 16 positions
    float4_t acc[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[t] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s4 = 0; s4 < 8; ++s4) {
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const float4 w = S.wa[(t * 8 + s4) * 64 + lane];
        acc[t] = mfma(w.x, x[4 * s4], acc[t]);
        acc[t] = mfma(w.y, x[4 * s4 + 1], acc[t]);
        acc[t] = mfma(w.z, x[4 * s4 + 2], acc[t]);
        acc[t] = mfma(w.w, x[4 * s4 + 3], acc[t]);
      }
    }
    // this lane holds R2 of row tk for groups 4 kk .. 4 kk + 3
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = 4 * kk + i;
      if (g < ng) {
        const float nrm = sqrtf(n2[i]);
        S.sc[wave][tk][g] = nrm > 0.f ? S.gs[g] / nrm : 0.f;
        if (valid)
          c.k_norms[row * kMaxGroups * cap + static_cast<size_t>(wp + r) * nslot + g] =
              __half_as_ushort(__float2half_rn(nrm));
      }
    }
    wave_sync();
    // codes of stream positions 16 t + 4 kk + i of row tk: one bit field
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int p0 = 16 * t + 4 * kk;
      uint32_t field = 0;
      int nb = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t pm = S.pm[p0 + i];
        const int b = (pm >> 10) & 15, g = (pm >> 14) & 7;
        const uint32_t code = scalar_code(S.thr + thr_index(b), b, acc[t][i] * S.sc[wave][tk][g]);
        field |= code << nb;
        nb += b;
      }
      const int bo = S.pm[p0] & 1023, w = bo >> 5, sh = bo & 31;
      if (valid) {
        atomicOr(&S.rw[wave][tk][w], field << sh);
        if (sh + nb > 32) atomicOr(&S.rw[wave][tk][w + 1], field >> (32 - sh));
      }
    }
    wave_sync();
    for (int idx = lane; idx < kSub * kw; idx += 64) {
      const int t2 = idx / kw, w = idx - t2 * kw;
      if (r0 + t2 < n_fit) c.k_codes[(row * cap + wp + r0 + t2) * kw + w] = S.rw[wave][t2][w];
      S.rw[wave][t2][w] = 0u;
    }
    wave_sync();
  }
}

// ---------------------------------------------------------------- values
// Workgroup bx of the value part: value tiles [bx T, bx T + T) of the rows
// the call touches, T = kWaves iters.  A wave owns whole 32-row value tiles;
// the words of a tile partly outside [write_pos, write_pos + n_new) keep the
// bits of the other rows.
template <bool BF16>
__device__ __forceinline__ void quant_values(LdsV& S, int bx, int iters, const Dims& d,
                                             const uint8_t* __restrict__ blob, const void* __restrict__ vin,
                                             int n_new, const int32_t* __restrict__ wpos, const CachePtrs& c) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.y, lz = blockIdx.z;
  const int layer = d.layer >= 0 ? d.layer : lz / d.batch;
  const int seq = lz % d.batch;
  const int cap = d.capacity, bv = d.v_bits;
  const int wp = wpos[seq];
  if (wp < 0 || wp >= cap) return;
  const int n_fit = min(n_new, cap - wp);
  const int tile0 = wp / kTile, n_tiles = (wp + n_fit - 1) / kTile - tile0 + 1;
  const int tw0 = bx * kWaves * iters;
  if (tw0 >= n_tiles) return;
  const int n_rows_blob = d.n_layers * d.n_kv;
  const float4* rsrc = reinterpret_cast<const float4*>(blob + layout_rotv_mfma_offset(n_rows_blob));
  const float* gthr = reinterpret_cast<const float*>(blob + kOffThr);
  for (int i = tid; i < kMatF4; i += kThreads) S.rb[i] = rsrc[i];
  for (int i = tid; i < kThresholdEntries; i += kThreads) S.thr[i] = gthr[i];
  __syncthreads();

  const int tk = lane & 15, kk = lane >> 4;
  const float* thr = S.thr + thr_index(bv);
  const float sq = sqrtf(static_cast<float>(kHeadDim));
  const size_t row = (static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + head;
  for (int it = 0; it < iters; ++it) {
    const int tw = tw0 + it * kWaves + wave;
    if (tw >= n_tiles) break;  // wave-uniform
    const int tile = tile0 + tw, P0 = tile * kTile;
    const int s_lo = max(P0, wp) - P0, s_hi = min(P0 + kTile, wp + n_fit) - P0;  // rows [s_lo, s_hi) are new
    uint32_t* gv = c.v_codes + (row * (cap / kTile) + tile) * kHeadDim * static_cast<size_t>(bv);
    const bool full = s_lo == 0 && s_hi == kTile;
    // tile words: zero, or the old words with the new rows' bits cleared
    for (int idx = lane; idx < kHeadDim * bv; idx += 64) {
      const int j = idx / bv, w = idx - j * bv;
      uint32_t old = 0u;
      if (!full) {
        const int lo_b = max(s_lo * bv - 32 * w, 0), hi_b = min(s_hi * bv - 32 * w, 32);
        const uint32_t mask = hi_b <= lo_b ? 0u : (hi_b - lo_b == 32 ? ~0u : ((1u << (hi_b - lo_b)) - 1u) << lo_b);
        old = gv[idx] & ~mask;
      }
      S.vt[wave][j][w] = old;
    }
#pragma unroll 1
    for (int h = 0; h < 2; ++h) {
      const int slot = 16 * h + tk;
      const bool valid = slot >= s_lo && slot < s_hi;
      float x[32];
      load_slice<BF16>(vin, ((static_cast<size_t>(lz) * n_new + (P0 + slot - wp)) * d.n_kv + head) * kHeadDim +
                                32 * kk,
                       valid, x);
      float ss = 0.f;
#pragma unroll
      for (int i = 0; i < 32; ++i) ss = fmaf(x[i], x[i], ss);
      ss += __shfl_xor(ss, 16, 64);
      ss += __shfl_xor(ss, 32, 64);
      const float nrm = sqrtf(ss);
      if (kk == 0) {
        S.nv[wave][slot] = nrm;
        if (valid) c.v_norms[row * cap + P0 + slot] = __half_as_ushort(__float2half_rn(nrm));
      }
      // Z[row][j] = sum_d x[row][d] Pi_V[j][d], 8 tiles of 16 coordinates
      float4_t acc[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) acc[t] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s4 = 0; s4 < 8; ++s4) {
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const float4 b = S.rb[(t * 8 + s4) * 64 + lane];
          acc[t] = mfma(x[4 * s4], b.x, acc[t]);
          acc[t] = mfma(x[4 * s4 + 1], b.y, acc[t]);
          acc[t] = mfma(x[4 * s4 + 2], b.z, acc[t]);
          acc[t] = mfma(x[4 * s4 + 3], b.w, acc[t]);
        }
      }
      wave_sync();
      // this lane: coordinate j = 16 t + tk of rows 16 h + 4 kk + i
      float scl[4];
      uint32_t keep = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int s = 16 * h + 4 * kk + i;
        const float n = S.nv[wave][s];
        scl[i] = n > 0.f ? sq / n : 0.f;
        keep |= (s >= s_lo && s < s_hi ? ((1u << bv) - 1u) : 0u) << (i * bv);
      }
      const int bit = (16 * h + 4 * kk) * bv, w = bit >> 5, sh = bit & 31;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        uint32_t field = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) field |= scalar_code(thr, bv, acc[t][i] * scl[i]) << (i * bv);
        field &= keep;
        const int j = 16 * t + tk;
        atomicOr(&S.vt[wave][j][w], field << sh);
        if (sh + 4 * bv > 32) atomicOr(&S.vt[wave][j][w + 1], field >> (32 - sh));
      }
      wave_sync();
    }
    for (int idx = lane; idx < kHeadDim * bv; idx += 64) gv[idx] = S.vt[wave][idx / bv][idx % bv];
    wave_sync();
  }
}

// One launch for both parts: workgroups [0, n_kwg) encode keys, the rest
// values; grid (n_kwg + n_vwg, n_kv, batch x layers in the call).
template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_quant_rows(Dims d, const uint8_t* __restrict__ blob,
                                                         const void* __restrict__ kin, const void* __restrict__ vin,
                                                         int n_new, const int32_t* __restrict__ wpos, CachePtrs c,
                                                         int n_kwg, int k_iters, int v_iters) {
  constexpr size_t kBytes = sizeof(LdsK) > sizeof(LdsV) ? sizeof(LdsK) : sizeof(LdsV);
  __shared__ __attribute__((aligned(16))) uint8_t smem[kBytes];
  const int bx = static_cast<int>(blockIdx.x);
  if (bx < n_kwg)
    quant_keys<BF16>(*reinterpret_cast<LdsK*>(smem), bx, k_iters, d, blob, kin, n_new, wpos, c);
  else
    quant_values<BF16>(*reinterpret_cast<LdsV*>(smem), bx - n_kwg, v_iters, d, blob, vin, n_new, wpos, c);
}

}  // namespace quant_detail

hipError_t launch_quantize_prefill(const Dims& d, const void* layout, const void* k, const void* v, int n_new,
                                   const int32_t* write_pos, const CachePtrs& c, hipStream_t s) {
  using namespace quant_detail;
  const uint8_t* blob = static_cast<const uint8_t*>(layout);
  const int lz = d.batch * d.n_lc;
  // rows per workgroup: small calls spread over more workgroups (one
  // sub-tile or value tile per wave), large ones amortise the 64 KB matrix
  // staged in LDS over more rows
  const long rows = static_cast<long>(n_new) * d.n_kv * lz;
  const int k_iters = rows <= 256L * 256 ? 1 : (rows <= 4L * 256 * 512 ? 2 : 4);
  const int v_iters = rows <= 256L * 512 ? 1 : 2;
  const int n_kwg = (n_new + kWaves * kSub * k_iters - 1) / (kWaves * kSub * k_iters);
  const int n_vwg = (n_new / kTile + 2 + kWaves * v_iters - 1) / (kWaves * v_iters);
  const dim3 grid(n_kwg + n_vwg, d.n_kv, lz);
  if (d.in_dtype == 1)
    hipLaunchKernelGGL(k_quant_rows<true>, grid, dim3(kThreads), 0, s, d, blob, k, v, n_new, write_pos, c, n_kwg,
                       k_iters, v_iters);
  else
    hipLaunchKernelGGL(k_quant_rows<false>, grid, dim3(kThreads), 0, s, d, blob, k, v, n_new, write_pos, c, n_kwg,
                       k_iters, v_iters);
  return hipGetLastError();
}

}  // namespace bgtq
