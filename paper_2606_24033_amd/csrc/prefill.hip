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
//  2. k_prefill_attn: the attention, 256 query rows per workgroup (8 waves of
//     32 rows, two 16-row column blocks per wave, so that each decoded
//     operand read from LDS feeds two MFMAs).  Decoded key tile: fp32 radius x centroid,
//     stored as fp16 hi + lo parts, so that hi/lo query x hi/lo key (three
//     MFMA passes, the lo x lo product left out) carries ~fp32 precision
//     through one full-width product per 32 coordinates; the value tile
//     holds the bare fp16 centroids (exact) and the value radius enters the
//     softmax weight.  Products run transposed, S^T = K Q^T and O^T = V^T P^T,
//     so that the softmax weights go from the S^T accumulators straight into
//     the B operand of the PV product (no trip through LDS).  The decoded
//     tiles are double-buffered: while a tile's products run, the same waves
//     decode the next tile into registers (independent of the products, so
//     its ALU work fills the MFMA latency) and store it into the other
//     buffer afterwards; one barrier per tile;
//  3. the same kernel's epilogue: out = Pi_V^T o, with fp32 MFMAs.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "layout.h"

namespace bgtq {
namespace prefill_detail {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;      // rotation kernel: 4 waves
constexpr int kAttnWaves = 8;  // attention kernel: 8 waves (2 per SIMD) ...
constexpr int kCB = 2;         // ... of 2 column blocks of 16 query rows
constexpr int kAttnThreads = kAttnWaves * 64;
constexpr int kRows = kAttnWaves * kCB * 16;  // query rows (position x head) per attention workgroup
// a thread's share of a tile's decode: kKPer stream positions of one key row
// (kKGrp threads per row) and kVPer tokens of one value dim (kVGrp threads
// per dim); kRawPer loads of each kind of raw word per thread
constexpr int kKPer = kKeyTile * kHeadDim / kAttnThreads, kKGrp = kHeadDim / kKPer;
constexpr int kVPer = kKeyTile * kHeadDim / kAttnThreads, kVGrp = kKeyTile / kVPer;
constexpr int kRawPer = (512 + kAttnThreads - 1) / kAttnThreads;
constexpr int kPieces = kKPer / 8 + kVPer / 8;  // decode pieces of 8 elements
constexpr int kQrotRows = 512;     // query rows (position x head) per rotation workgroup
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();

// ---- LDS map of the attention kernel (bytes)
constexpr int kKStride = 136;  // halves per decoded key row (128 + 8 pad)
constexpr int kVStride = 68;   // halves per decoded value row (64 + 4 pad: conflict-free stores and PV reads)
// decoded tile (two buffers): key hi, key lo [64 tokens][kKStride] fp16,
// values [128 dims][kVStride] fp16, value radii [64] fp16
constexpr int kDecKH = 0;
constexpr int kDecKL = kDecKH + 64 * kKStride * 2;
constexpr int kDecV = kDecKL + 64 * kKStride * 2;
constexpr int kDecVN = kDecV + 128 * kVStride * 2;
constexpr int kDecBytes = kDecVN + 64 * 2;
// raw tile (two buffers): key words [64][k_words], value words [2 value
// tiles][128 dims][b_V] (the second tile kRawV1 words further), key radii
// [64][8] fp16, value radii [64] fp16
constexpr int kRawK = 0;
constexpr int kRawV = kRawK + 64 * kMaxKWords * 4;
constexpr int kRawV1 = 4;  // words between the two value tiles: their same dims on other banks
constexpr int kRawKN = kRawV + (2 * kHeadDim * 8 + kRawV1) * 4;
constexpr int kRawVN = kRawKN + 64 * 8 * 2;
constexpr int kRawBytes = kRawVN + 64 * 2;
constexpr int kOffDec = 0;
constexpr int kOffRaw = kOffDec + 2 * kDecBytes;
constexpr int kOffCb = kOffRaw + 2 * kRawBytes;  // fp16 codebooks
constexpr int kOffMeta = kOffCb + 1024;          // per position: bit offset | b << 10 | group << 14 | table << 17
constexpr int kTileLds = kOffMeta + 512;
constexpr int kRotVLds = kHeadDim * kHeadDim * 4;  // Pi_V staged for the epilogue
constexpr int kLdsBytes = kTileLds > kRotVLds ? kTileLds : kRotVLds;
static_assert(kLdsBytes <= 160 * 1024, "LDS of one workgroup");
static_assert(kDecBytes % 16 == 0 && kRawBytes % 16 == 0, "16-byte aligned buffers");
static_assert(2 * kCodebookEntries <= 1024, "codebook staging");
static_assert(kKeyTile * kMaxKWords / 4 <= kRawPer * kAttnThreads && 2 * kHeadDim * 8 / 4 <= kRawPer * kAttnThreads &&
                  kKeyTile * 8 <= kRawPer * kAttnThreads && kKeyTile <= kAttnThreads,
              "raw loads of a tile");
static_assert(kKPer % 8 == 0 && kVPer % 8 == 0 && kVPer <= kTile, "decode pieces inside one value tile");

// Load of a T at a 32-bit byte offset from a wave-uniform base (the global
// load form with a scalar base and a 32-bit vector offset).
template <class T>
__device__ __forceinline__ T ld_at(const void* base, uint32_t byte_off) {
  return *reinterpret_cast<const T*>(static_cast<const char*>(base) + byte_off);
}

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
// grid (ceil(n_q G / kQrotRows), n_kv, batch).  qr: [batch][n_q][Hq][128]
// fp32.  The rotation of a query row is one product with a 128 x 128 matrix
// in stream order, W[p][k] = log2 e / sqrt(d_g d_h) Pi_g[j][k - g_pos] for
// p = g_pos + j and k in the same group g (zero elsewhere), applied to the
// row gathered into stream order.  W is staged in LDS once per workgroup
// (transposed, Wt[k][p]); each wave multiplies 16-row tiles by it with fp32
// MFMAs (16x16x4: 32 steps of 4 coordinates x 8 tiles of 16 outputs).
__global__ __launch_bounds__(kThreads) void k_prefill_qrot(Dims d, const uint8_t* __restrict__ blob,
                                                           const void* __restrict__ q, int n_q,
                                                           float* __restrict__ qr) {
  __shared__ float wt[kHeadDim * kHeadDim];                  // Wt[k][p]
  __shared__ float qs[kThreads / 64][16][kHeadDim + 4];      // per wave: 16 rows in stream order
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kvh = blockIdx.y, seq = blockIdx.z;
  const int G = d.group, hq = d.n_kv * G;
  const int n_rows_blob = d.n_layers * d.n_kv;
  const RowMeta* M = reinterpret_cast<const RowMeta*>(blob + kOffRows) + (d.layer * d.n_kv + kvh);
  const float* rowrot = reinterpret_cast<const float*>(blob + layout_rowrot_offset(n_rows_blob)) +
                        static_cast<size_t>(d.layer * d.n_kv + kvh) * kRowRotFloats;
  for (int i = tid; i < kHeadDim * kHeadDim; i += kThreads) wt[i] = 0.f;
  __syncthreads();
  {
    // column p (thread & 127) of Wt: the rotation row j = p - g_pos of its group
    const int p = tid & 127;
    const int g = M->grp[p], p0 = M->g_pos[g], dg = M->g_dim[g], j = p - p0;
    int off = 0;
    for (int e = 0; e < g; ++e) off += M->g_dim[e] * M->g_dim[e];
    const float scale = kLog2e * rsqrtf(static_cast<float>(dg) * kHeadDim);
    for (int k = tid >> 7; k < dg; k += kThreads / kHeadDim)
      wt[(p0 + k) * kHeadDim + p] = rowrot[off + k * dg + j] * scale;  // Pi_dg transposed: [k dg + j] = Pi[j][k]
  }
  const int dimk = M->dim[lane], dimk2 = M->dim[lane + 64];  // stream position -> source dim
  __syncthreads();
  const int nr = n_q * G;
  const int r_wg = blockIdx.x * kQrotRows;
  float (*qw)[kHeadDim + 4] = qs[wave];
  for (int t0 = r_wg + wave * 16; t0 < min(r_wg + kQrotRows, nr); t0 += kThreads / 4) {
    // gather 16 rows into stream order (rows past the end are zero)
    for (int r = 0; r < 16; ++r) {
      const int row = t0 + r;
      float a = 0.f, b = 0.f;
      if (row < nr) {
        const int i = row / G, h = row - (row / G) * G;
        const size_t base = ((static_cast<size_t>(seq) * n_q + i) * hq + kvh * G + h) * kHeadDim;
        a = ld_q(q, base + dimk, d.in_dtype);
        b = ld_q(q, base + dimk2, d.in_dtype);
      }
      qw[r][lane] = a;
      qw[r][lane + 64] = b;
    }
    // one wave writes and reads its own rows: LDS operations of a wave
    // complete in order, so only the compiler must keep the order
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
    float4_t acc[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[t] = float4_t{0.f, 0.f, 0.f, 0.f};
    const int ar = lane & 15, ak = lane >> 4;
#pragma unroll 4
    for (int st = 0; st < kHeadDim / 4; ++st) {
      const float a = qw[ar][4 * st + ak];
      const float* wrow = wt + (4 * st + ak) * kHeadDim + ar;
#pragma unroll
      for (int t = 0; t < 8; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, wrow[16 * t], acc[t], 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = t0 + 4 * ak + i;
      if (row < nr) {
        const int qi = row / G, h = row - (row / G) * G;
        float* dst = qr + ((static_cast<size_t>(seq) * n_q + qi) * hq + kvh * G + h) * kHeadDim + ar;
#pragma unroll
        for (int t = 0; t < 8; ++t) dst[16 * t] = acc[t][i];
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");  // reads of these rows before the next tile's writes
    __builtin_amdgcn_wave_barrier();
  }
}

// ---------------------------------------------------------------- 2. attention
// Lane roles in the products (16x16x32 f16 MFMAs; l16 = lane % 16, g4 =
// lane / 16): the A operand comes from the decoded tile (token or dim l16 of
// a 16-block, 8 consecutive k from 8 g4), the B operand is one of the wave's
// kCB column blocks of 16 query rows (row l16, the same k), and an
// accumulator holds tokens (S^T) or dims (O^T) 4 g4 .. +3 of its block for
// row l16.

// A thread's share of the decode of a tile, stored into decoded buffer dec:
// keys of token tid / kKGrp, stream positions kKPer (tid % kKGrp) + E0 .. +7
// (fp32 radius x centroid split into fp16 hi and lo parts).  The code's next
// word may belong to the next row or lie past the tile's words: it is in
// LDS, and only used when the field straddles.
template <int E0>
__device__ __forceinline__ void decode_keys(const uint8_t* smem, const uint8_t* raw, uint8_t* dec, int tid, int kw) {
  const int t = tid / kKGrp, pq = (tid % kKGrp) * kKPer + E0;
  const uint32_t* meta = reinterpret_cast<const uint32_t*>(smem + kOffMeta) + pq;
  const uint32_t* kr = reinterpret_cast<const uint32_t*>(raw + kRawK) + t * kw;
  const uint16_t* knrm = reinterpret_cast<const uint16_t*>(raw + kRawKN) + t * 8;
  const uint16_t* cbs = reinterpret_cast<const uint16_t*>(smem + kOffCb);
  half8_t hv, lv;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t m = meta[e];
    const uint32_t off = m & 1023u, b = (m >> 10) & 15u;
    const uint32_t w = off >> 5;
    const uint32_t code = __builtin_amdgcn_alignbit(kr[w + 1], kr[w], off & 31u) & ((1u << b) - 1u);
    const float x = h2f(knrm[(m >> 14) & 7u]) * h2f(cbs[(m >> 17) + code]);
    const _Float16 xh = static_cast<_Float16>(x);
    hv[e] = xh;
    lv[e] = static_cast<_Float16>(x - static_cast<float>(xh));
  }
  *reinterpret_cast<half8_t*>(reinterpret_cast<_Float16*>(dec + kDecKH) + t * kKStride + pq) = hv;
  *reinterpret_cast<half8_t*>(reinterpret_cast<_Float16*>(dec + kDecKL) + t * kKStride + pq) = lv;
}
// Values of dim tid / kVGrp, tokens kVPer (tid % kVGrp) + E0 .. +7 of the
// tile (codes LSB-first in the dim's b_V words of its 32-token value tile),
// stored into dec; the first piece also copies the tile's value radii.
template <int E0>
__device__ __forceinline__ void decode_values(const uint8_t* smem, const uint8_t* raw, uint8_t* dec, int tid,
                                              int bv) {
  const int vd = tid / kVGrp, vq = (tid % kVGrp) * kVPer + E0;
  const uint32_t* vr =
      reinterpret_cast<const uint32_t*>(raw + kRawV) + ((vq / kTile) * kHeadDim + vd) * bv + (vq / kTile) * kRawV1;
  const uint16_t* cb = reinterpret_cast<const uint16_t*>(smem + kOffCb) + cb_index(bv);
  const uint32_t mask = (1u << bv) - 1u;
  half8_t hv;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t bit = static_cast<uint32_t>(((vq % kTile) + e) * bv);
    const uint32_t w = bit >> 5;
    const uint32_t code = __builtin_amdgcn_alignbit(vr[w + 1], vr[w], bit & 31u) & mask;
    hv[e] = __builtin_bit_cast(_Float16, cb[code]);
  }
  // two 8-byte stores: the row stride keeps only 8-byte alignment
  uint2* dst = reinterpret_cast<uint2*>(reinterpret_cast<_Float16*>(dec + kDecV) + vd * kVStride + vq);
  const uint4 hb = __builtin_bit_cast(uint4, hv);
  dst[0] = make_uint2(hb.x, hb.y);
  dst[1] = make_uint2(hb.z, hb.w);
  if (E0 == 0 && tid < kKeyTile)
    reinterpret_cast<uint16_t*>(dec + kDecVN)[tid] = reinterpret_cast<const uint16_t*>(raw + kRawVN)[tid];
}
// Decode pieces P0 .. P1 - 1 (the key pieces first, then the value pieces).
template <int P0, int P1>
__device__ __forceinline__ void decode_pieces(const uint8_t* smem, const uint8_t* raw, uint8_t* dec, int tid, int kw,
                                              int bv) {
  if constexpr (P0 < P1) {
    if constexpr (P0 < kKPer / 8)
      decode_keys<8 * P0>(smem, raw, dec, tid, kw);
    else
      decode_values<8 * (P0 - kKPer / 8)>(smem, raw, dec, tid, bv);
    decode_pieces<P0 + 1, P1>(smem, raw, dec, tid, kw, bv);
  }
}

// S^T of the 32-token half HH of the tile in dec for every column block.
template <int HH>
__device__ __forceinline__ void qk_half(const uint8_t* dec, int l16, int g4, const half8_t (&qh)[kCB][4],
                                        const half8_t (&ql)[kCB][4], float4_t (&s)[kCB][2]) {
  const _Float16* khi = reinterpret_cast<const _Float16*>(dec + kDecKH);
  const _Float16* klo = reinterpret_cast<const _Float16*>(dec + kDecKL);
#pragma unroll
  for (int jj = 0; jj < 2; ++jj) {
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) s[cb][jj] = float4_t{0.f, 0.f, 0.f, 0.f};
    const int kbase = (32 * HH + 16 * jj + l16) * kKStride + 8 * g4;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const half8_t ah = *reinterpret_cast<const half8_t*>(khi + kbase + 32 * ks);
      const half8_t al = *reinterpret_cast<const half8_t*>(klo + kbase + 32 * ks);
#pragma unroll
      for (int cb = 0; cb < kCB; ++cb) {
        s[cb][jj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, qh[cb][ks], s[cb][jj], 0, 0, 0);
        s[cb][jj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(al, qh[cb][ks], s[cb][jj], 0, 0, 0);
        s[cb][jj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, ql[cb][ks], s[cb][jj], 0, 0, 0);
      }
    }
  }
}

// Causal mask and online-softmax update of half HH (base 2; one row per
// lane column), then O^T += V^T P^T over the 8 blocks of 16 dims.  The mask
// is applied only where a token of the half can lie past a row of the wave
// (pos_min = the wave's first position; the tiles before it need none).
// exp2 is the hardware instruction: its arguments are <= 0 here and a result
// below the normal range (flushed to 0) is negligible beside the sum.
template <int HH>
__device__ __forceinline__ void softmax_pv_half(const uint8_t* dec, int t0, int l16, int g4, const int (&pos)[kCB],
                                                int pos_min, float4_t (&s)[kCB][2], float (&m_run)[kCB],
                                                float (&l_run)[kCB], float4_t (&o)[kCB][8]) {
  const uint16_t* vnrm = reinterpret_cast<const uint16_t*>(dec + kDecVN);
  const uint2 va = *reinterpret_cast<const uint2*>(vnrm + 32 * HH + 4 * g4);
  const uint2 vb = *reinterpret_cast<const uint2*>(vnrm + 32 * HH + 16 + 4 * g4);
  const uint32_t vr[4] = {va.x, va.y, vb.x, vb.y};
  half8_t pb[kCB];  // B operand of O^T = V^T P^T: tokens {4 g4 + i, 16 + 4 g4 + i} of the half
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
    if (t0 + 32 * HH + 31 > pos_min) {
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tok = t0 + 32 * HH + 16 * jj + 4 * g4 + i;
          s[cb][jj][i] = tok > pos[cb] ? kNegInf : s[cb][jj][i];
        }
    }
    float mx = kNegInf;
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[cb][jj][i]);
    mx = max4g(mx);
    // m_run stays -inf only while every token so far is masked (tokens past pos)
    const float mn = fmaxf(m_run[cb], mx);
    const float corr = m_run[cb] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m_run[cb] - mn);
    const float mref = mn == kNegInf ? 0.f : mn;
    m_run[cb] = mn;
    float ps = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float p = __builtin_amdgcn_exp2f(s[cb][e >> 2][e & 3] - mref);
      ps += p;
      const uint16_t nb = static_cast<uint16_t>(vr[e >> 1] >> (16 * (e & 1)));
      pb[cb][e] = static_cast<_Float16>(p * h2f(nb));
    }
    l_run[cb] = l_run[cb] * corr + ps;
    // the accumulators are rescaled only when a running maximum of the wave
    // moved (rare after the first tiles)
    if (__builtin_amdgcn_ballot_w64(corr != 1.f) != 0) {
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) o[cb][cc] *= corr;
    }
  }
  const _Float16* vh = reinterpret_cast<const _Float16*>(dec + kDecV);
#pragma unroll
  for (int cc = 0; cc < 8; ++cc) {
    const _Float16* vrow = vh + (16 * cc + l16) * kVStride + 32 * HH + 4 * g4;
    const uint2 a0 = *reinterpret_cast<const uint2*>(vrow);
    const uint2 a1 = *reinterpret_cast<const uint2*>(vrow + 16);
    const half8_t a = __builtin_bit_cast(half8_t, make_uint4(a0.x, a0.y, a1.x, a1.y));
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb)
      o[cb][cc] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, pb[cb], o[cb][cc], 0, 0, 0);
  }
}

// grid (n_tiles, n_kv, batch), tiles in reverse order (the longest first).
__global__ __launch_bounds__(kAttnThreads) void k_prefill_attn(
    Dims d, const uint8_t* __restrict__ blob, const float* __restrict__ qr, int n_q,
    const int32_t* __restrict__ q_pos0, int max_pos, CachePtrs c, float* __restrict__ out) {
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

  // this lane's query rows (column l16 of the wave's column blocks): query
  // position index ri, head rh (recomputed where needed, to save registers)
  const auto row_of = [&](int cb, int& ri, int& rh) {
    const int r = qt * kRows + (wave * kCB + cb) * 16 + l16;
    ri = r / G;
    rh = r - ri * G;
  };
  int pos[kCB];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
    int ri, rh;
    row_of(cb, ri, rh);
    pos[cb] = max(0, min(pos0 + min(ri, n_q - 1), max_pos));
  }
  // the wave's first (smallest) position: its first row
  const int pos_min = max(0, min(pos0 + min((qt * kRows + wave * kCB * 16) / G, n_q - 1), max_pos));
  // the tile's last position bounds its key loop
  const int i_last = min(n_q - 1, (qt * kRows + kRows - 1) / G);
  const int pos_last = max(0, min(pos0 + i_last, max_pos));
  const int n_kt = pos_last / kKeyTile + 1;

  // query operands (B of S^T = K Q^T): dims 32 ks + 8 g4 .. +7 of the row,
  // fp16 hi and lo parts
  half8_t qh[kCB][4], ql[kCB][4];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
    int ri, rh;
    row_of(cb, ri, rh);
    const bool valid = ri < n_q;
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
        qh[cb][ks][e] = h;
        ql[cb][ks][e] = static_cast<_Float16>(x - static_cast<float>(h));
      }
    }
  }
  // per-position decode metadata and the codebooks
  uint16_t* cbs = reinterpret_cast<uint16_t*>(smem + kOffCb);
  uint32_t* meta = reinterpret_cast<uint32_t*>(smem + kOffMeta);
  for (int i = tid; i < kCodebookEntries; i += kAttnThreads) cbs[i] = c16[i];
  if (tid < kHeadDim) {
    const uint32_t b = M->width[tid];
    meta[tid] = static_cast<uint32_t>(M->bitoff[tid]) | (b << 10) | (static_cast<uint32_t>(M->grp[tid]) << 14) |
                (static_cast<uint32_t>(cb_index(static_cast<int>(b))) << 17);
  }

  const size_t row = (static_cast<size_t>(d.layer) * d.batch + seq) * d.n_kv + kvh;
  const uint32_t* kc = c.k_codes + row * cap * kw;
  const uint16_t* kn = c.k_norms + row * kMaxGroups * cap;
  const uint32_t* vc = c.v_codes + row * (cap / kTile) * kHeadDim * bv;
  const uint16_t* vnp = c.v_norms + row * cap;

  float m_run[kCB], l_run[kCB];
  float4_t o[kCB][8];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
    m_run[cb] = kNegInf;
    l_run[cb] = 0.f;
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) o[cb][cc] = float4_t{0.f, 0.f, 0.f, 0.f};
  }

  // Raw words of one tile, loaded into registers while the previous tile is
  // processed: kRawPer 16-byte loads of key words (64 k_words words in all)
  // and of value words (2 x 128 x b_V) per thread, kRawPer key radii and
  // one value radius; every load in bounds (offsets clamped), stored only
  // where it exists.
  const int nk4 = kKeyTile * kw / 4, nv4 = 2 * kHeadDim * bv / 4, nkn = kKeyTile * nslot;
  uint4 pk[kRawPer], pv[kRawPer];
  uint16_t pkn[kRawPer], pvn;
  const auto load_raw = [&](int ta) {
    const uint32_t* ks = kc + static_cast<size_t>(ta) * kw;
    const uint32_t* vs = vc + static_cast<size_t>(ta / kTile) * kHeadDim * bv;  // two value tiles, contiguous
    const uint16_t* ns = kn + static_cast<size_t>(ta) * nslot;
#pragma unroll
    for (int j = 0; j < kRawPer; ++j) {
      const int i = tid + j * kAttnThreads;
      // opaque offsets: keeps the scalar-base + 32-bit-offset load form
      uint32_t o0 = 16u * min(i, nk4 - 1), o1 = 16u * min(i, nv4 - 1), o2 = 2u * min(i, nkn - 1);
      asm volatile("" : "+v"(o0), "+v"(o1), "+v"(o2));
      pk[j] = ld_at<uint4>(ks, o0);
      pv[j] = ld_at<uint4>(vs, o1);
      pkn[j] = ld_at<uint16_t>(ns, o2);
    }
    uint32_t o3 = 2u * min(tid, kKeyTile - 1);
    asm volatile("" : "+v"(o3));
    pvn = ld_at<uint16_t>(vnp + ta, o3);
  };
  const auto store_raw = [&](uint8_t* raw) {
#pragma unroll
    for (int j = 0; j < kRawPer; ++j) {
      const int i = tid + j * kAttnThreads;
      if (i < nk4) reinterpret_cast<uint4*>(raw + kRawK)[i] = pk[j];
      if (i < nv4) reinterpret_cast<uint4*>(raw + kRawV)[i + (4 * i >= kHeadDim * bv ? kRawV1 / 4 : 0)] = pv[j];
      if (i < nkn) reinterpret_cast<uint16_t*>(raw + kRawKN)[(i / nslot) * 8 + i % nslot] = pkn[j];
    }
    if (tid < kKeyTile) reinterpret_cast<uint16_t*>(raw + kRawVN)[tid] = pvn;
  };
  uint8_t* const dec0 = smem + kOffDec;
  uint8_t* const raw0 = smem + kOffRaw;

  // Pipeline: tile kt's products run on decoded buffer kt % 2 while tile
  // kt + 1 is decoded from raw buffer (kt + 1) % 2 into decoded buffer
  // (kt + 1) % 2, and tile kt + 2's raw words are in flight to registers.
  // The one barrier per tile separates every buffer's writes from its reads
  // (raw buffer r is written two tiles after its decode was read, decoded
  // buffer b one tile after its products).  The decode after the last tile
  // reads stale LDS words into a buffer nobody reads (all its addresses are
  // in range).
  load_raw(0);
  store_raw(raw0);
  if (n_kt > 1) load_raw(kKeyTile);
  __syncthreads();
  decode_pieces<0, kPieces>(smem, raw0, dec0, tid, kw, bv);
  for (int kt = 0; kt < n_kt; ++kt) {
    const int t0 = kt * kKeyTile;  // t0 + 63 < capacity (a multiple of 64, above pos_last)
    const uint8_t* const dcur = dec0 + (kt & 1) * kDecBytes;
    uint8_t* const dnxt = dec0 + ((kt + 1) & 1) * kDecBytes;
    uint8_t* const rnxt = raw0 + ((kt + 1) & 1) * kRawBytes;
    if (kt + 1 < n_kt) store_raw(rnxt);
    if (kt + 2 < n_kt) load_raw(t0 + 2 * kKeyTile);
    __syncthreads();

    // the next tile's decode, a quarter of its pieces beside each product
    // phase (independent of the products: its ALU work and LDS latency fill
    // the MFMA time; sched_barrier keeps the phases apart, hoisted together
    // their LDS reads would hold registers that the products need)
    constexpr int q1 = kPieces / 4, q2 = kPieces / 2, q3 = 3 * kPieces / 4;
    float4_t s[kCB][2];
    decode_pieces<0, q1>(smem, rnxt, dnxt, tid, kw, bv);
    __builtin_amdgcn_sched_barrier(0);
    qk_half<0>(dcur, l16, g4, qh, ql, s);
    __builtin_amdgcn_sched_barrier(0);
    decode_pieces<q1, q2>(smem, rnxt, dnxt, tid, kw, bv);
    __builtin_amdgcn_sched_barrier(0);
    softmax_pv_half<0>(dcur, t0, l16, g4, pos, pos_min, s, m_run, l_run, o);
    __builtin_amdgcn_sched_barrier(0);
    decode_pieces<q2, q3>(smem, rnxt, dnxt, tid, kw, bv);
    __builtin_amdgcn_sched_barrier(0);
    qk_half<1>(dcur, l16, g4, qh, ql, s);
    __builtin_amdgcn_sched_barrier(0);
    decode_pieces<q3, kPieces>(smem, rnxt, dnxt, tid, kw, bv);
    __builtin_amdgcn_sched_barrier(0);
    softmax_pv_half<1>(dcur, t0, l16, g4, pos, pos_min, s, m_run, l_run, o);
  }

  // ---- epilogue: o / (l sqrt(d_h)), then out = Pi_V^T o (fp32 MFMAs over Pi_V staged in LDS)
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
    const float lt = sum4g(l_run[cb]);
    // the codes' 1/sqrt(d_h) (value radius n_V over sqrt(d_h) times a unit-variance centroid)
    const float inv = lt > 0.f ? 0.08838834764831845f / lt : 0.f;
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) o[cb][cc] *= inv;
  }
  __syncthreads();
  float* rv = reinterpret_cast<float*>(smem);
  {
    const float4* src = reinterpret_cast<const float4*>(blob + kOffRotV);
    for (int i = tid; i < kHeadDim * kHeadDim / 4; i += kAttnThreads) reinterpret_cast<float4*>(rv)[i] = src[i];
  }
  __syncthreads();
#pragma unroll 1
  for (int c2 = 0; c2 < 8; ++c2) {
    float4_t acc[kCB];
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) acc[cb] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cc = 0; cc < 8; ++cc)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // A[d'][k] = Pi_V[16 cc + 4 k + i][d'], B[k][row] = o[cc][i] of lane group k
        const float a = rv[(16 * cc + 4 * g4 + i) * kHeadDim + 16 * c2 + l16];
#pragma unroll
        for (int cb = 0; cb < kCB; ++cb)
          acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, o[cb][cc][i], acc[cb], 0, 0, 0);
      }
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) {
      int ri, rh;
      row_of(cb, ri, rh);
      if (ri < n_q) {
        float* dst = out + ((static_cast<size_t>(seq) * n_q + ri) * hq + kvh * G + rh) * kHeadDim;
        *reinterpret_cast<float4*>(dst + 16 * c2 + 4 * g4) = make_float4(acc[cb][0], acc[cb][1], acc[cb][2], acc[cb][3]);
      }
    }
  }
}

}  // namespace prefill_detail

hipError_t launch_prefill_attn(const Dims& d, const void* layout, const void* q, int n_q,
                               const int32_t* q_pos0, int max_pos, const CachePtrs& c, float* qr_ws,
                               float* out, hipStream_t s) {
  using namespace prefill_detail;
  const uint8_t* blob = static_cast<const uint8_t*>(layout);
  dim3 g1((n_q * d.group + kQrotRows - 1) / kQrotRows, d.n_kv, d.batch);
  hipLaunchKernelGGL(k_prefill_qrot, g1, dim3(kThreads), 0, s, d, blob, q, n_q, qr_ws);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int n_tiles = (n_q * d.group + kRows - 1) / kRows;
  dim3 g2(n_tiles, d.n_kv, d.batch);
  hipLaunchKernelGGL(k_prefill_attn, g2, dim3(kAttnThreads), 0, s, d, blob, qr_ws, n_q, q_pos0, max_pos, c, out);
  return hipGetLastError();
}

}  // namespace bgtq
