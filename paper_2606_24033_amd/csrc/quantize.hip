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

// Workgroups of W waves: 16 for long appends (the 64 KB matrix staged in LDS
// serves more rows), 4 for calls of up to 64K rows, which then spread over
// more CUs: two such workgroups fit a CU (under 80 KB of LDS each), and a
// value tile is split between two waves.  (A 16-wave value workgroup of 16
// tiles keeps each SIMD's MFMA pipe busy ~30 us on its own, with most CUs
// idle in a short call.)
constexpr int kWavesLong = 16, kWavesShort = 4;
constexpr int kSub = 16;                          // rows per wave sub-tile (one MFMA column block)
constexpr int kMatF4 = kMfmaMatFloats / 4;        // float4 entries of one MFMA-order matrix

template <int W>
struct LdsK {
  float4 wa[kMatF4];                          // the row's W, A operand order
  float4 ma[W == kWavesLong ? 8 * 64 : 1];    // group membership, A operand order ([s4][lane]);
                                              // the short path keeps it in registers
  uint32_t rw[W][kSub][kMaxKWords];           // per wave: packed key rows
  float sc[W][kSub][kMaxGroups];              // per wave: sqrt(d_g) / radius of each row and group
  float thr[kThresholdEntries];
  uint32_t pm[kHeadDim];                      // per stream position: bit offset | b << 10 | group << 14
  float gs[kMaxGroups];                       // sqrt(d_g)
  uint8_t gd[kHeadDim];                       // group ordinal of each input dim
};
template <int W>
struct LdsV {
  float4 rb[kMatF4];                          // Pi_V, B operand order
  uint32_t vt[W][kHeadDim][8];                // per wave: words of one value tile
  float nv[W][32];                            // per wave: the tile's value radii
  float thr[kThresholdEntries];
};
// Short calls: a value tile is shared by two waves (16 rows each), two tiles
// per 4-wave workgroup.
struct LdsVS {
  float4 rb[kMatF4];                          // Pi_V, B operand order
  uint32_t vt[kWavesShort / 2][kHeadDim][8];  // per tile: its words
  float nv[kWavesShort / 2][32];              // per tile: its value radii
  float thr[kThresholdEntries];
};
static_assert(sizeof(LdsK<kWavesLong>) <= 160 * 1024 && sizeof(LdsV<kWavesLong>) <= 160 * 1024, "LDS of one workgroup");
// two short-call workgroups share a CU
static_assert(sizeof(LdsK<kWavesShort>) <= 80 * 1024 && sizeof(LdsVS) <= 80 * 1024, "LDS of a short-call workgroup");

// Copy of the 64 KB MFMA-order matrix into LDS with every global load issued
// before the first store (a loop of load-store pairs waits out one memory
// latency per round: 16 rounds in a 4-wave workgroup).
template <int W>
__device__ __forceinline__ void stage_matrix(float4* dst, const float4* __restrict__ src, int tid) {
  constexpr int kPer = kMatF4 / (W * 64);
  static_assert(kMatF4 % (W * 64) == 0, "matrix staging");
  float4 t[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) t[u] = src[tid + u * W * 64];
#pragma unroll
  for (int u = 0; u < kPer; ++u) dst[tid + u * W * 64] = t[u];
}

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
// W kSub iters.
template <bool BF16, int W>
__device__ __forceinline__ void quant_keys(LdsK<W>& S, int bx, int iters, const Dims& d,
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
  constexpr int kThreads = W * 64;
  const int r_wg = bx * W * kSub * iters;
  if (r_wg >= n_fit) return;
  const int n_rows_blob = d.n_layers * d.n_kv;
  const int ri = layer * d.n_kv + head;
  const RowMeta* M = reinterpret_cast<const RowMeta*>(blob + kOffRows) + ri;
  const float4* wsrc = reinterpret_cast<const float4*>(blob + layout_kdense_offset(n_rows_blob)) +
                       static_cast<size_t>(ri) * kMatF4;
  const float* gthr = reinterpret_cast<const float*>(blob + kOffThr);
  const int ng = M->n_groups;

  stage_matrix<W>(S.wa, wsrc, tid);
  for (int i = tid; i < W * kSub * kMaxKWords; i += kThreads) (&S.rw[0][0][0])[i] = 0u;
  for (int i = tid; i < kThresholdEntries; i += kThreads) S.thr[i] = gthr[i];
  if (tid < kHeadDim) {
    const int g = M->grp[tid];
    S.gd[M->dim[tid]] = static_cast<uint8_t>(g);
    S.pm[tid] = static_cast<uint32_t>(M->bitoff[tid]) | (static_cast<uint32_t>(M->width[tid]) << 10) |
                (static_cast<uint32_t>(g) << 14);
  }
  if (tid < kMaxGroups) S.gs[tid] = tid < ng ? sqrtf(static_cast<float>(M->g_dim[tid])) : 0.f;
  __syncthreads();
  float mreg[32];  // short path: this lane's membership entries (unused in the long path)
  if constexpr (W == kWavesLong) {
    for (int i = tid; i < 8 * 64; i += kThreads) {
      const int s4 = i >> 6, l = i & 63, g = l & 15, d0 = 32 * (l >> 4) + 4 * s4;
      S.ma[i] = make_float4(S.gd[d0] == g ? 1.f : 0.f, S.gd[d0 + 1] == g ? 1.f : 0.f, S.gd[d0 + 2] == g ? 1.f : 0.f,
                            S.gd[d0 + 3] == g ? 1.f : 0.f);
    }
    __syncthreads();
  } else {
    const int g = lane & 15, d0 = 32 * (lane >> 4);
#pragma unroll
    for (int j = 0; j < 32; ++j) mreg[j] = S.gd[d0 + j] == g ? 1.f : 0.f;
  }

  const int tk = lane & 15, kk = lane >> 4;
  const int kw = d.k_words, nslot = (ng + 1) & ~1;
  const size_t row = (static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + head;
  for (int it = 0; it < iters; ++it) {
    const int r0 = r_wg + (it * W + wave) * kSub;
    if (r0 >= n_fit) break;  // wave-uniform
    const int r = r0 + tk;
    const bool valid = r < n_fit;
    float x[32];
    load_slice<BF16>(kin, ((static_cast<size_t>(lz) * n_new + r) * d.n_kv + head) * kHeadDim + 32 * kk, valid, x);

    // group radii: R2[g][row] = sum_d [group(d) = g] x[row][d]^2
    float4_t n2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s4 = 0; s4 < 8; ++s4) {
      float4 m;
      if constexpr (W == kWavesLong) m = S.ma[s4 * 64 + lane];
      else m = make_float4(mreg[4 * s4], mreg[4 * s4 + 1], mreg[4 * s4 + 2], mreg[4 * s4 + 3]);
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
// the call touches, T = W iters.  A wave owns whole 32-row value tiles;
// the words of a tile partly outside [write_pos, write_pos + n_new) keep the
// bits of the other rows.
template <bool BF16, int W>
__device__ __forceinline__ void quant_values(LdsV<W>& S, int bx, int iters, const Dims& d,
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
  constexpr int kThreads = W * 64;
  const int tw0 = bx * W * iters;
  if (tw0 >= n_tiles) return;
  const int n_rows_blob = d.n_layers * d.n_kv;
  const float4* rsrc = reinterpret_cast<const float4*>(blob + layout_rotv_mfma_offset(n_rows_blob));
  const float* gthr = reinterpret_cast<const float*>(blob + kOffThr);
  stage_matrix<W>(S.rb, rsrc, tid);
  for (int i = tid; i < kThresholdEntries; i += kThreads) S.thr[i] = gthr[i];
  __syncthreads();

  const int tk = lane & 15, kk = lane >> 4;
  const float* thr = S.thr + thr_index(bv);
  const float sq = sqrtf(static_cast<float>(kHeadDim));
  const size_t row = (static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + head;
  for (int it = 0; it < iters; ++it) {
    const int tw = tw0 + it * W + wave;
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

// Short calls: workgroup bx encodes value tiles 2 bx and 2 bx + 1 of the
// rows the call touches; waves 2 u and 2 u + 1 take rows 0-15 and 16-31 of
// tile 2 bx + u and assemble its words together in LDS.
template <bool BF16>
__device__ __forceinline__ void quant_values_short(LdsVS& S, int bx, const Dims& d, const uint8_t* __restrict__ blob,
                                                   const void* __restrict__ vin, int n_new,
                                                   const int32_t* __restrict__ wpos, const CachePtrs& c) {
  constexpr int W = kWavesShort, kThreads = W * 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.y, lz = blockIdx.z;
  const int layer = d.layer >= 0 ? d.layer : lz / d.batch;
  const int seq = lz % d.batch;
  const int cap = d.capacity, bv = d.v_bits;
  const int wp = wpos[seq];
  if (wp < 0 || wp >= cap) return;  // (uniform over the workgroup: before any barrier)
  const int n_fit = min(n_new, cap - wp);
  const int tile0 = wp / kTile, n_tiles = (wp + n_fit - 1) / kTile - tile0 + 1;
  const int tw0 = bx * (W / 2);
  if (tw0 >= n_tiles) return;
  const int n_rows_blob = d.n_layers * d.n_kv;
  const float4* rsrc = reinterpret_cast<const float4*>(blob + layout_rotv_mfma_offset(n_rows_blob));
  const float* gthr = reinterpret_cast<const float*>(blob + kOffThr);
  stage_matrix<W>(S.rb, rsrc, tid);
  for (int i = tid; i < kThresholdEntries; i += kThreads) S.thr[i] = gthr[i];

  const int u = wave >> 1, h = wave & 1;  // the wave's tile of the workgroup and its half
  const int tile = tile0 + tw0 + u, P0 = tile * kTile;
  const bool active = tw0 + u < n_tiles;  // the same for both waves of a tile
  const int s_lo = max(P0, wp) - P0, s_hi = min(P0 + kTile, wp + n_fit) - P0;  // rows [s_lo, s_hi) are new
  const size_t row = (static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + head;
  uint32_t* gv = c.v_codes + (row * (cap / kTile) + tile) * kHeadDim * static_cast<size_t>(bv);
  if (active) {
    // tile words: zero, or the old words with the new rows' bits cleared
    const bool full = s_lo == 0 && s_hi == kTile;
    for (int idx = 64 * h + lane; idx < kHeadDim * bv; idx += 128) {
      const int j = idx / bv, w = idx - j * bv;
      uint32_t old = 0u;
      if (!full) {
        const int lo_b = max(s_lo * bv - 32 * w, 0), hi_b = min(s_hi * bv - 32 * w, 32);
        const uint32_t mask = hi_b <= lo_b ? 0u : (hi_b - lo_b == 32 ? ~0u : ((1u << (hi_b - lo_b)) - 1u) << lo_b);
        old = gv[idx] & ~mask;
      }
      S.vt[u][j][w] = old;
    }
  }
  __syncthreads();  // matrix, thresholds and the tile words
  if (active) {
    const int tk = lane & 15, kk = lane >> 4;
    const float* thr = S.thr + thr_index(bv);
    const float sq = sqrtf(static_cast<float>(kHeadDim));
    const int slot = 16 * h + tk;
    const bool valid = slot >= s_lo && slot < s_hi;
    float x[32];
    load_slice<BF16>(vin, ((static_cast<size_t>(lz) * n_new + (P0 + slot - wp)) * d.n_kv + head) * kHeadDim + 32 * kk,
                     valid, x);
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < 32; ++i) ss = fmaf(x[i], x[i], ss);
    ss += __shfl_xor(ss, 16, 64);
    ss += __shfl_xor(ss, 32, 64);
    const float nrm = sqrtf(ss);
    if (kk == 0) {
      S.nv[u][slot] = nrm;
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
    wave_sync();  // this half's radii (written by this wave)
    // this lane: coordinate j = 16 t + tk of rows 16 h + 4 kk + i
    float scl[4];
    uint32_t keep = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 16 * h + 4 * kk + i;
      const float n = S.nv[u][r];
      scl[i] = n > 0.f ? sq / n : 0.f;
      keep |= (r >= s_lo && r < s_hi ? ((1u << bv) - 1u) : 0u) << (i * bv);
    }
    const int bit = (16 * h + 4 * kk) * bv, w = bit >> 5, sh = bit & 31;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      uint32_t field = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) field |= scalar_code(thr, bv, acc[t][i] * scl[i]) << (i * bv);
      field &= keep;
      const int j = 16 * t + tk;
      atomicOr(&S.vt[u][j][w], field << sh);
      if (sh + 4 * bv > 32) atomicOr(&S.vt[u][j][w + 1], field >> (32 - sh));
    }
  }
  __syncthreads();  // both halves' bits are in the tile words
  if (active)
    for (int idx = 64 * h + lane; idx < kHeadDim * bv; idx += 128) gv[idx] = S.vt[u][idx / bv][idx % bv];
}

// One launch for both parts; grid (n_kwg + n_vwg, n_kv, batch x layers in
// the call).  16-wave workgroups: [0, n_kwg) encode keys, the rest values.
// 4-wave workgroups (short calls, two per CU): the value workgroups come
// first, so that the key workgroups fill in behind.
template <bool BF16, int W>
__global__ __launch_bounds__(W * 64) void k_quant_rows(Dims d, const uint8_t* __restrict__ blob,
                                                        const void* __restrict__ kin, const void* __restrict__ vin,
                                                        int n_new, const int32_t* __restrict__ wpos, CachePtrs c,
                                                        int n_kwg, int n_vwg, int k_iters, int v_iters) {
  constexpr size_t kVBytes = W == kWavesLong ? sizeof(LdsV<W>) : sizeof(LdsVS);
  constexpr size_t kBytes = sizeof(LdsK<W>) > kVBytes ? sizeof(LdsK<W>) : kVBytes;
  __shared__ __attribute__((aligned(16))) uint8_t smem[kBytes];
  const int bx = static_cast<int>(blockIdx.x);
  const bool keys = W == kWavesLong ? bx < n_kwg : bx >= n_vwg;
  if (keys)
    quant_keys<BF16, W>(*reinterpret_cast<LdsK<W>*>(smem), W == kWavesLong ? bx : bx - n_vwg, k_iters, d, blob, kin,
                        n_new, wpos, c);
  else if constexpr (W == kWavesLong)
    quant_values<BF16, W>(*reinterpret_cast<LdsV<W>*>(smem), bx - n_kwg, v_iters, d, blob, vin, n_new, wpos, c);
  else
    quant_values_short<BF16>(*reinterpret_cast<LdsVS*>(smem), bx, d, blob, vin, n_new, wpos, c);
}

}  // namespace quant_detail

hipError_t launch_quantize_prefill(const Dims& d, const void* layout, const void* k, const void* v, int n_new,
                                   const int32_t* write_pos, const CachePtrs& c, hipStream_t s) {
  using namespace quant_detail;
  const uint8_t* blob = static_cast<const uint8_t*>(layout);
  const int lz = d.batch * d.n_lc;
  // rows per workgroup: small calls spread over more workgroups (one
  // sub-tile or value tile per wave, 4-wave workgroups up to 64K rows), large
  // ones amortise the 64 KB matrix staged in LDS over more rows
  const long rows = static_cast<long>(n_new) * d.n_kv * lz;
  const int k_iters = rows <= 256L * 256 ? 1 : (rows <= 4L * 256 * 512 ? 2 : 4);
  const int v_iters = rows <= 256L * 512 ? 1 : 2;
  const auto go = [&](auto kern, int w) {
    const int n_kwg = (n_new + w * kSub * k_iters - 1) / (w * kSub * k_iters);
    // value tiles per workgroup: w v_iters (a wave per tile), or 2 (short calls)
    const int vt_wg = w == kWavesLong ? w * v_iters : kWavesShort / 2;
    const int n_vwg = (n_new / kTile + 2 + vt_wg - 1) / vt_wg;
    const dim3 grid(n_kwg + n_vwg, d.n_kv, lz);
    hipLaunchKernelGGL(kern, grid, dim3(w * 64), 0, s, d, blob, k, v, n_new, write_pos, c, n_kwg, n_vwg, k_iters,
                       v_iters);
  };
  const bool bf = d.in_dtype == 1, short_call = rows <= 256L * 256;
  if (short_call) {
    if (bf) go(k_quant_rows<true, kWavesShort>, kWavesShort);
    else go(k_quant_rows<false, kWavesShort>, kWavesShort);
  } else {
    if (bf) go(k_quant_rows<true, kWavesLong>, kWavesLong);
    else go(k_quant_rows<false, kWavesLong>, kWavesLong);
  }
  return hipGetLastError();
}

}  // namespace bgtq
