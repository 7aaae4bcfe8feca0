// Causal prefill attention over the packed cache (Sec. 4, prefill paragraph):
// each workgroup owns a tile of query rows, streams the packed K/V tiles of
// its (layer, sequence, KV head) up to the tile's last position, decodes each
// tile once into LDS for all of its query rows, and accumulates QK^T and PV
// with a causal mask under an online softmax.  No fp16 cache and no attention
// matrix is written.
//
// Three launches on the caller's stream:
//  1. k_prefill_qrot: the Q-side rotation of every query row into the key
//     stream order, qr[p] = log2 e (Pi_g q_g)_j / sqrt(d_g d_h) at stream
//     position p = g_pos[g] + j (fp32, into the caller's workspace);
//  2. k_prefill_attn: the attention, 64 query rows per workgroup (4 waves of
//     16 rows).  Decoded key tile: fp32 radius x centroid, stored as fp16 hi
//     + lo parts, so that hi/lo query x hi/lo key (three MFMA passes, the
//     lo x lo product left out) carries ~fp32 precision through one
//     full-width product per 32 coordinates; the value tile holds the bare
//     fp16 centroids (exact) and the value radius enters the softmax weight.
//     Products run transposed, S^T = K Q^T and O^T = V^T P^T, so that the
//     softmax weights go from the S^T accumulators straight into the B
//     operand of the PV product (no trip through LDS);
//  3. the same kernel's epilogue: out = Pi_V^T o, with fp32 MFMAs.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "layout.h"

namespace bgtq {
namespace prefill_detail {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;  // 4 waves
constexpr int kRows = 64;      // query rows (position x head) per attention workgroup
constexpr int kQrotPos = 8;    // query positions per rotation workgroup
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();

// ---- LDS map of the attention kernel (bytes)
constexpr int kKStride = 136;                  // halves per decoded key row (128 + 8 pad)
constexpr int kVStride = 72;                   // halves per decoded value row (64 + 8 pad)
constexpr int kOffKH = 0;                      // [64 tokens][kKStride] fp16 hi
constexpr int kOffKL = kOffKH + 64 * kKStride * 2;   // lo
constexpr int kOffVH = kOffKL + 64 * kKStride * 2;   // [128 dims][kVStride] fp16
constexpr int kOffKRaw = kOffVH + 128 * kVStride * 2;  // [64][k_words] uint32
constexpr int kOffKNrm = kOffKRaw + 64 * kMaxKWords * 4;  // [64][8] fp16 group radii
constexpr int kOffVNrm = kOffKNrm + 64 * 8 * 2;           // [64] fp16
constexpr int kOffCb = kOffVNrm + 64 * 2;                 // fp16 codebooks
constexpr int kOffMeta = kOffCb + 1024;                   // bitoff u16[128], width u8[128], grp u8[128]
constexpr int kOffVRaw = kOffMeta + 512;                  // [2 value tiles][128 dims][b_V] uint32
constexpr int kTileLds = kOffVRaw + 2 * kHeadDim * 8 * 4;
constexpr int kRotVLds = kHeadDim * kHeadDim * 4;         // Pi_V staged for the epilogue
constexpr int kLdsBytes = kTileLds > kRotVLds ? kTileLds : kRotVLds;
static_assert(kLdsBytes <= 80 * 1024, "two workgroups per CU");
static_assert(2 * kCodebookEntries <= 1024, "codebook staging");

__device__ __forceinline__ float h2f(uint16_t b) { return static_cast<float>(__builtin_bit_cast(_Float16, b)); }

// max / sum over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (the lanes that hold
// the same query row of an MFMA accumulator); gfx950 lane swaps
__device__ __forceinline__ void swap16(float v, float& r0, float& r1) {
  unsigned x = __builtin_bit_cast(unsigned, v), y = x;
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1\n\ts_nop 1" : "+v"(x), "+v"(y));
  r0 = __builtin_bit_cast(float, x);
  r1 = __builtin_bit_cast(float, y);
}
__device__ __forceinline__ void swap32(float v, float& r0, float& r1) {
  unsigned x = __builtin_bit_cast(unsigned, v), y = x;
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(x), "+v"(y));
  r0 = __builtin_bit_cast(float, x);
  r1 = __builtin_bit_cast(float, y);
}
__device__ __forceinline__ float max4g(float v) {
  float a, b;
  swap16(v, a, b);
  swap32(fmaxf(a, b), a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float sum4g(float v) {
  float a, b;
  swap16(v, a, b);
  swap32(a + b, a, b);
  return a + b;
}

__device__ __forceinline__ float ld_q(const void* q, size_t i, int in_dtype) {  // BGTQ_BF16 = 1
  if (in_dtype == 1) {
    const uint16_t b = static_cast<const uint16_t*>(q)[i];
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
  }
  return static_cast<const float*>(q)[i];
}

// ---------------------------------------------------------------- 1. rotation
// grid (ceil(n_q / kQrotPos), n_kv, batch).  qr: [batch][n_q][Hq][128] fp32.
__global__ __launch_bounds__(kThreads) void k_prefill_qrot(Dims d, const uint8_t* __restrict__ blob,
                                                           const void* __restrict__ q, int n_q,
                                                           float* __restrict__ qr) {
  __shared__ float rs[kRowRotFloats];                // the row's group rotations (transposed blocks)
  __shared__ float qs[kQrotPos * 8 * kHeadDim];      // the queries in stream order
  const int tid = threadIdx.x;
  const int kvh = blockIdx.y, seq = blockIdx.z, i0 = blockIdx.x * kQrotPos;
  const int G = d.group, hq = d.n_kv * G;
  const int n_rows_blob = d.n_layers * d.n_kv;
  const RowMeta* M = reinterpret_cast<const RowMeta*>(blob + kOffRows) + (d.layer * d.n_kv + kvh);
  const float* rowrot = reinterpret_cast<const float*>(blob + layout_rowrot_offset(n_rows_blob)) +
                        static_cast<size_t>(d.layer * d.n_kv + kvh) * kRowRotFloats;
  const int ng = M->n_groups;
  int rtot = 0;
  for (int g = 0; g < ng; ++g) rtot += M->g_dim[g] * M->g_dim[g];
  for (int i = tid; i < rtot; i += kThreads) rs[i] = rowrot[i];
  const int npos = min(kQrotPos, n_q - i0);
  for (int e = tid; e < npos * G * kHeadDim; e += kThreads) {
    const int r = e >> 7, p = e & 127;  // r = position-in-block * G + head
    const int i = i0 + r / G, h = r - (r / G) * G;
    const size_t src = ((static_cast<size_t>(seq) * n_q + i) * hq + kvh * G + h) * kHeadDim + M->dim[p];
    qs[e] = ld_q(q, src, d.in_dtype);
  }
  __syncthreads();
  const int p = tid & 127;
  const int g = M->grp[p], p0 = M->g_pos[g], dg = M->g_dim[g], j = p - p0;
  int off = 0;
  for (int e = 0; e < g; ++e) off += M->g_dim[e] * M->g_dim[e];
  const float* rt = rs + off;  // Pi_dg transposed: rt[k dg + j] = Pi[j][k]
  const float scale = kLog2e * rsqrtf(static_cast<float>(dg) * kHeadDim);
  for (int r = tid >> 7; r < npos * G; r += kThreads / kHeadDim) {
    const float* qq = qs + r * kHeadDim + p0;
    float a0 = 0.f, a1 = 0.f;
    int k = 0;
    for (; k + 2 <= dg; k += 2) {
      a0 = fmaf(rt[k * dg + j], qq[k], a0);
      a1 = fmaf(rt[(k + 1) * dg + j], qq[k + 1], a1);
    }
    const int i = i0 + r / G, h = r - (r / G) * G;
    qr[((static_cast<size_t>(seq) * n_q + i) * hq + kvh * G + h) * kHeadDim + p] = (a0 + a1) * scale;
  }
}

// ---------------------------------------------------------------- 2. attention
// grid (n_tiles, n_kv, batch), tiles in reverse order (the longest first).
__global__ __launch_bounds__(kThreads, 2) void k_prefill_attn(Dims d, const uint8_t* __restrict__ blob,
                                                              const float* __restrict__ qr, int n_q,
                                                              const int32_t* __restrict__ q_pos0, int max_pos,
                                                              CachePtrs c, float* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g4 = lane >> 4, l16 = lane & 15;
  const int n_tiles = gridDim.x;
  const int qt = n_tiles - 1 - static_cast<int>(blockIdx.x);
  const int kvh = blockIdx.y, seq = blockIdx.z;
  const int G = d.group, hq = d.n_kv * G, cap = d.capacity, kw = d.k_words, bv = d.v_bits;
  const RowMeta* M = reinterpret_cast<const RowMeta*>(blob + kOffRows) + (d.layer * d.n_kv + kvh);
  const uint16_t* c16 = reinterpret_cast<const uint16_t*>(blob + kOffC16);
  const int ng = M->n_groups;
  const int nslot = (ng + 1) & ~1;
  const int pos0 = q_pos0[seq];

  // this lane's query row (column l16 of the wave's accumulators)
  const int r = qt * kRows + wave * 16 + l16;
  const int ri = r / G, rh = r - ri * G;
  const bool valid = ri < n_q;
  const int pos = max(0, min(pos0 + min(ri, n_q - 1), max_pos));
  // the tile's last position bounds its key loop
  const int i_last = min(n_q - 1, (qt * kRows + kRows - 1) / G);
  const int pos_last = max(0, min(pos0 + i_last, max_pos));
  const int n_kt = pos_last / kKeyTile + 1;

  // query operand (B of S^T = K Q^T): dims 32 ks + 8 g4 .. +7 of the row, hi and lo
  half8_t qh[4], ql[4];
  {
    const float* src = qr + ((static_cast<size_t>(seq) * n_q + min(ri, n_q - 1)) * hq + kvh * G + rh) * kHeadDim;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const float4 a = *reinterpret_cast<const float4*>(src + 32 * ks + 8 * g4);
      const float4 b = *reinterpret_cast<const float4*>(src + 32 * ks + 8 * g4 + 4);
      const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = valid ? v[e] : 0.f;
        const _Float16 h = static_cast<_Float16>(x);
        qh[ks][e] = h;
        ql[ks][e] = static_cast<_Float16>(x - static_cast<float>(h));
      }
    }
  }
  // per-position decode metadata and the codebooks
  uint16_t* cbs = reinterpret_cast<uint16_t*>(smem + kOffCb);
  uint16_t* mbit = reinterpret_cast<uint16_t*>(smem + kOffMeta);
  uint8_t* mwid = smem + kOffMeta + 256;
  uint8_t* mgrp = smem + kOffMeta + 384;
  for (int i = tid; i < kCodebookEntries; i += kThreads) cbs[i] = c16[i];
  if (tid < kHeadDim) {
    mbit[tid] = M->bitoff[tid];
    mwid[tid] = M->width[tid];
    mgrp[tid] = M->grp[tid];
  }

  const size_t row = (static_cast<size_t>(d.layer) * d.batch + seq) * d.n_kv + kvh;
  const uint32_t* kc = c.k_codes + row * cap * kw;
  const uint16_t* kn = c.k_norms + row * kMaxGroups * cap;
  const uint32_t* vc = c.v_codes + row * (cap / kTile) * kHeadDim * bv;
  const uint16_t* vnp = c.v_norms + row * cap;
  uint32_t* kraw = reinterpret_cast<uint32_t*>(smem + kOffKRaw);
  uint16_t* knrm = reinterpret_cast<uint16_t*>(smem + kOffKNrm);
  uint16_t* vnrm = reinterpret_cast<uint16_t*>(smem + kOffVNrm);
  uint32_t* vraw = reinterpret_cast<uint32_t*>(smem + kOffVRaw);
  _Float16* khi = reinterpret_cast<_Float16*>(smem + kOffKH);
  _Float16* klo = reinterpret_cast<_Float16*>(smem + kOffKL);
  _Float16* vh = reinterpret_cast<_Float16*>(smem + kOffVH);

  float m_run = kNegInf, l_run = 0.f;
  float4_t o[8];
#pragma unroll
  for (int cc = 0; cc < 8; ++cc) o[cc] = float4_t{0.f, 0.f, 0.f, 0.f};

  for (int kt = 0; kt < n_kt; ++kt) {
    const int t0 = kt * kKeyTile;  // t0 + 63 < capacity (a multiple of 64, above pos_last)
    __syncthreads();               // the previous tile's operands are consumed
    // ---- raw tile to LDS: key words and radii, value words and radii
    for (int i = tid; i < kKeyTile * kw; i += kThreads) kraw[i] = kc[static_cast<size_t>(t0) * kw + i];
    for (int i = tid; i < 2 * kHeadDim * bv; i += kThreads)  // two 32-token value tiles, contiguous
      vraw[i] = vc[static_cast<size_t>(t0 / kTile) * kHeadDim * bv + i];
    for (int i = tid; i < kKeyTile * nslot; i += kThreads) {
      const int t = i / nslot, gg = i - t * nslot;
      knrm[t * 8 + gg] = kn[static_cast<size_t>(t0) * nslot + i];
    }
    if (tid < kKeyTile) vnrm[tid] = vnp[t0 + tid];
    __syncthreads();
    // ---- decode the key tile: token t, stream positions 32 pq .. +31
    {
      const int t = tid >> 2, pq = (tid & 3) * 32;
      const uint32_t* kr = kraw + t * kw;
#pragma unroll 4
      for (int e8 = 0; e8 < 4; ++e8) {
        half8_t hv, lv;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int p = pq + 8 * e8 + e;
          const int off = mbit[p], b = mwid[p], gg = mgrp[p];
          const int w = off >> 5, sh = off & 31;
          const uint32_t lo = kr[w];
          const uint32_t hi = sh + b > 32 ? kr[w + 1] : 0u;
          const uint32_t code = static_cast<uint32_t>(((static_cast<uint64_t>(hi) << 32) | lo) >> sh) & ((1u << b) - 1u);
          const float x = h2f(knrm[t * 8 + gg]) * h2f(cbs[cb_index(b) + code]);
          const _Float16 xh = static_cast<_Float16>(x);
          hv[e] = xh;
          lv[e] = static_cast<_Float16>(x - static_cast<float>(xh));
        }
        *reinterpret_cast<half8_t*>(khi + t * kKStride + pq + 8 * e8) = hv;
        *reinterpret_cast<half8_t*>(klo + t * kKStride + pq + 8 * e8) = lv;
      }
    }
    // ---- decode the value tile: dim vd, tokens 32 vhalf .. +31 (codes LSB-first
    // in the dim's b_V words of its 32-token tile)
    {
      const int vd = tid >> 1, vhalf = tid & 1;
      const uint32_t* vr = vraw + (vhalf * kHeadDim + vd) * bv;
      const uint16_t* cb = cbs + cb_index(bv);
      const uint32_t mask = (1u << bv) - 1u;
#pragma unroll
      for (int e8 = 0; e8 < 4; ++e8) {
        half8_t hv;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int bit = (8 * e8 + e) * bv, w = bit >> 5, sh = bit & 31;
          const uint32_t lo = vr[w];
          const uint32_t hi = sh + bv > 32 ? vr[w + 1] : 0u;
          const uint32_t code = static_cast<uint32_t>(((static_cast<uint64_t>(hi) << 32) | lo) >> sh) & mask;
          hv[e] = __builtin_bit_cast(_Float16, cb[code]);
        }
        *reinterpret_cast<half8_t*>(vh + vd * kVStride + 32 * vhalf + 8 * e8) = hv;
      }
    }
    __syncthreads();

    // ---- S^T = K Q^T: 4 tiles of 16 tokens; lane holds tokens 4 g4 + i of tile j, row l16
    float4_t s[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float4_t acc = {0.f, 0.f, 0.f, 0.f};
      const int kbase = (16 * j + l16) * kKStride + 8 * g4;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const half8_t ah = *reinterpret_cast<const half8_t*>(khi + kbase + 32 * ks);
        const half8_t al = *reinterpret_cast<const half8_t*>(klo + kbase + 32 * ks);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, qh[ks], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(al, qh[ks], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, ql[ks], acc, 0, 0, 0);
      }
      s[j] = acc;
    }
    // ---- causal mask and online softmax (base 2; one row per lane column)
    float mx = kNegInf;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tok = t0 + 16 * j + 4 * g4 + i;
        s[j][i] = tok > pos ? kNegInf : s[j][i];
        mx = fmaxf(mx, s[j][i]);
      }
    mx = max4g(mx);
    const float mn = fmaxf(m_run, mx);  // finite from the first tile on (token 0 <= pos)
    const float corr = m_run == kNegInf ? 0.f : exp2f(m_run - mn);
    m_run = mn;
    float ps = 0.f;
    half8_t pb[2];  // B operand of O^T = V^T P^T: tokens {4 g4 + i, 16 + 4 g4 + i} of each 32-token step
#pragma unroll
    for (int sstep = 0; sstep < 2; ++sstep) {
      const uint2 va = *reinterpret_cast<const uint2*>(vnrm + 32 * sstep + 4 * g4);
      const uint2 vb = *reinterpret_cast<const uint2*>(vnrm + 32 * sstep + 16 + 4 * g4);
      const uint32_t vr[4] = {va.x, va.y, vb.x, vb.y};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = exp2f(s[2 * sstep + (e >> 2)][e & 3] - mn);
        ps += p;
        const uint16_t nb = static_cast<uint16_t>(vr[e >> 1] >> (16 * (e & 1)));
        pb[sstep][e] = static_cast<_Float16>(p * h2f(nb));
      }
    }
    l_run = l_run * corr + ps;
    if (corr != 1.f) {
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) o[cc] *= corr;
    }
    // ---- O^T += V^T P^T: 8 tiles of 16 dims; lane holds dims 4 g4 + i of tile cc, row l16
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) {
      const _Float16* vrow = vh + (16 * cc + l16) * kVStride + 4 * g4;
#pragma unroll
      for (int sstep = 0; sstep < 2; ++sstep) {
        const uint2 a0 = *reinterpret_cast<const uint2*>(vrow + 32 * sstep);
        const uint2 a1 = *reinterpret_cast<const uint2*>(vrow + 32 * sstep + 16);
        const uint4 u = make_uint4(a0.x, a0.y, a1.x, a1.y);
        o[cc] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, u), pb[sstep], o[cc], 0, 0, 0);
      }
    }
  }

  // ---- epilogue: o / (l sqrt(d_h)), then out = Pi_V^T o (fp32 MFMAs over Pi_V staged in LDS)
  const float lt = sum4g(l_run);
  // the codes' 1/sqrt(d_h) (value radius n_V over sqrt(d_h) times a unit-variance centroid)
  const float inv = lt > 0.f ? 0.08838834764831845f / lt : 0.f;
#pragma unroll
  for (int cc = 0; cc < 8; ++cc) o[cc] *= inv;
  __syncthreads();
  float* rv = reinterpret_cast<float*>(smem);
  {
    const float4* src = reinterpret_cast<const float4*>(blob + kOffRotV);
    for (int i = tid; i < kHeadDim * kHeadDim / 4; i += kThreads) reinterpret_cast<float4*>(rv)[i] = src[i];
  }
  __syncthreads();
  float* dst = out + ((static_cast<size_t>(seq) * n_q + min(ri, n_q - 1)) * hq + kvh * G + rh) * kHeadDim;
#pragma unroll 1
  for (int c2 = 0; c2 < 8; ++c2) {
    float4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cc = 0; cc < 8; ++cc)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // A[d'][k] = Pi_V[16 cc + 4 k + i][d'], B[k][row] = o[cc][i] of lane group k
        const float a = rv[(16 * cc + 4 * g4 + i) * kHeadDim + 16 * c2 + l16];
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, o[cc][i], acc, 0, 0, 0);
      }
    if (valid) *reinterpret_cast<float4*>(dst + 16 * c2 + 4 * g4) = make_float4(acc[0], acc[1], acc[2], acc[3]);
  }
}

}  // namespace prefill_detail

hipError_t launch_prefill_attn(const Dims& d, const void* layout, const void* q, int n_q,
                               const int32_t* q_pos0, int max_pos, const CachePtrs& c, float* qr_ws,
                               float* out, hipStream_t s) {
  using namespace prefill_detail;
  const uint8_t* blob = static_cast<const uint8_t*>(layout);
  dim3 g1((n_q + kQrotPos - 1) / kQrotPos, d.n_kv, d.batch);
  hipLaunchKernelGGL(k_prefill_qrot, g1, dim3(kThreads), 0, s, d, blob, q, n_q, qr_ws);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int n_tiles = (n_q * d.group + kRows - 1) / kRows;
  dim3 g2(n_tiles, d.n_kv, d.batch);
  hipLaunchKernelGGL(k_prefill_attn, g2, dim3(kThreads), 0, s, d, blob, qr_ws, n_q, q_pos0, max_pos, c, out);
  return hipGetLastError();
}

}  // namespace bgtq
