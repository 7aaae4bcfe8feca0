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
//  2. k_prefill_attn: the attention, 256 query rows per workgroup (16 waves
//     of 16 rows), so that each decoded tile serves 256 rows.  Decoded key tile: fp32 radius x centroid, stored as fp16 hi
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

constexpr int kThreads = 256;       // rotation kernel: 4 waves
constexpr int kAttnThreads = 1024;  // attention kernel: 16 waves of 16 query rows
constexpr int kRows = 256;          // query rows (position x head) per attention workgroup
constexpr int kQrotRows = 512;       // query rows (position x head) per rotation workgroup
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
constexpr int kOffMeta = kOffCb + 1024;                   // per position: bit offset | b << 10 | group << 14 | table << 17
constexpr int kOffVRaw = kOffMeta + 512;                  // [2 value tiles][128 dims][b_V] uint32
constexpr int kOffQLo = kOffVRaw + 2 * kHeadDim * 8 * 4;   // [16 waves][4 steps][64 lanes] x 8 fp16: query lo parts
constexpr int kTileLds = kOffQLo + 16 * 4 * 64 * 16;
constexpr int kRotVLds = kHeadDim * kHeadDim * 4;         // Pi_V staged for the epilogue
constexpr int kLdsBytes = kTileLds > kRotVLds ? kTileLds : kRotVLds;
static_assert(kLdsBytes <= 160 * 1024, "LDS of one workgroup");
static_assert(2 * kCodebookEntries <= 1024, "codebook staging");

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
// grid (n_tiles, n_kv, batch), tiles in reverse order (the longest first).
__global__ __launch_bounds__(kAttnThreads) void k_prefill_attn(Dims d, const uint8_t* __restrict__ blob,
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

  // query operand (B of S^T = K Q^T): dims 32 ks + 8 g4 .. +7 of the row, hi
  // parts in registers, lo parts in LDS (registers are the limit here)
  half8_t qh[4];
  half8_t* qlo = reinterpret_cast<half8_t*>(smem + kOffQLo) + wave * 4 * 64 + lane;
  {
    const float* src = qr + ((static_cast<size_t>(seq) * n_q + min(ri, n_q - 1)) * hq + kvh * G + rh) * kHeadDim;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const float4 a = *reinterpret_cast<const float4*>(src + 32 * ks + 8 * g4);
      const float4 b = *reinterpret_cast<const float4*>(src + 32 * ks + 8 * g4 + 4);
      const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
      half8_t lo;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = valid ? v[e] : 0.f;
        const _Float16 h = static_cast<_Float16>(x);
        qh[ks][e] = h;
        lo[e] = static_cast<_Float16>(x - static_cast<float>(h));
      }
      qlo[ks * 64] = lo;
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

  // Raw words of one tile, one or two per thread (at most 2048 key words,
  // 2048 value words, 512 key radii, 64 value radii); every load in bounds
  // (indices clamped), stored only where they exist.
  const int nk = kKeyTile * kw, nv = 2 * kHeadDim * bv;
  const int nr_t = tid / nslot;
  // per-thread byte offsets of the loads (clamped into the tile)
  const uint32_t ok0 = 4u * min(tid, nk - 1), ok1 = 4u * min(tid + kAttnThreads, nk - 1);
  const uint32_t ov0 = 4u * min(tid, nv - 1), ov1 = 4u * min(tid + kAttnThreads, nv - 1);
  const uint32_t okn = 2u * min(tid, kKeyTile * nslot - 1), ovn = 2u * min(tid, kKeyTile - 1);
  uint32_t pk0, pk1, pv0, pv1;
  uint16_t pkn, pvn;
  const auto load_raw = [&](int ta) {
    const uint32_t* ks = kc + static_cast<size_t>(ta) * kw;
    const uint32_t* vs = vc + static_cast<size_t>(ta / kTile) * kHeadDim * bv;  // two value tiles, contiguous
    const uint16_t* ns = kn + static_cast<size_t>(ta) * nslot;
    // opaque offsets: keeps the scalar-base + 32-bit-offset load form instead
    // of per-lane 64-bit pointers carried across iterations
    uint32_t o0 = ok0, o1 = ok1, o2 = ov0, o3 = ov1, o4 = okn, o5 = ovn;
    asm volatile("" : "+v"(o0), "+v"(o1), "+v"(o2), "+v"(o3), "+v"(o4), "+v"(o5));
    pk0 = ld_at<uint32_t>(ks, o0);
    pk1 = ld_at<uint32_t>(ks, o1);
    pv0 = ld_at<uint32_t>(vs, o2);
    pv1 = ld_at<uint32_t>(vs, o3);
    pkn = ld_at<uint16_t>(ns, o4);
    pvn = ld_at<uint16_t>(vnp + ta, o5);
  };
  load_raw(0);
  for (int kt = 0; kt < n_kt; ++kt) {
    const int t0 = kt * kKeyTile;  // t0 + 63 < capacity (a multiple of 64, above pos_last)
    __syncthreads();               // the previous tile's operands are consumed
    // ---- raw tile to LDS: key words and radii, value words and radii
    // this tile's raw words (loaded during the previous tile) to LDS, then
    // the next tile's loads, in flight during this tile's decode and products
    if (tid < nk) kraw[tid] = pk0;
    if (tid + kAttnThreads < nk) kraw[tid + kAttnThreads] = pk1;
    if (tid < nv) vraw[tid] = pv0;
    if (tid + kAttnThreads < nv) vraw[tid + kAttnThreads] = pv1;
    if (tid < kKeyTile * nslot) knrm[nr_t * 8 + (tid - nr_t * nslot)] = pkn;
    if (tid < kKeyTile) vnrm[tid] = pvn;
    if (kt + 1 < n_kt) load_raw(t0 + kKeyTile);
    __syncthreads();
    // ---- decode the key tile: token t, stream positions pq .. pq + 7
    {
      const int t = tid >> 4, pq = (tid & 15) * 8;
      const uint32_t* kr = kraw + t * kw;
      half8_t hv, lv;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t mt = meta[pq + e];
        const uint32_t off = mt & 1023u, b = (mt >> 10) & 15u;
        // the code's word and the next (the next may belong to the next row
        // or lie past the tile's words: in LDS, and unused then)
        const uint32_t w = off >> 5;
        const uint32_t code = __builtin_amdgcn_alignbit(kr[w + 1], kr[w], off & 31u) & ((1u << b) - 1u);
        const float x = h2f(knrm[t * 8 + ((mt >> 14) & 7u)]) * h2f(cbs[(mt >> 17) + code]);
        const _Float16 xh = static_cast<_Float16>(x);
        hv[e] = xh;
        lv[e] = static_cast<_Float16>(x - static_cast<float>(xh));
      }
      *reinterpret_cast<half8_t*>(khi + t * kKStride + pq) = hv;
      *reinterpret_cast<half8_t*>(klo + t * kKStride + pq) = lv;
    }
    // ---- decode the value tile: dim vd, tokens 8 vq .. 8 vq + 7 (codes LSB-first
    // in the dim's b_V words of its 32-token tile)
    {
      const int vd = tid >> 3, vq = tid & 7;
      const uint32_t* vr = vraw + ((vq >> 2) * kHeadDim + vd) * bv;
      const uint16_t* cb = cbs + cb_index(bv);
      const uint32_t mask = (1u << bv) - 1u;
      half8_t hv;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t bit = static_cast<uint32_t>((8 * (vq & 3) + e) * bv);
        const uint32_t w = bit >> 5;
        // (the next word may lie past the dim's words: in LDS, and unused then)
        const uint32_t code = __builtin_amdgcn_alignbit(vr[w + 1], vr[w], bit & 31u) & mask;
        hv[e] = __builtin_bit_cast(_Float16, cb[code]);
      }
      *reinterpret_cast<half8_t*>(vh + vd * kVStride + 8 * vq) = hv;
    }
    __syncthreads();

    // Two 32-token halves, each: S^T = K Q^T over 2 tiles of 16 tokens (lane
    // holds tokens 4 g4 + i of tile j, row l16), the causal mask and an
    // online-softmax update (base 2; one row per lane column), then
    // O^T += V^T P^T over 8 tiles of 16 dims (lane holds dims 4 g4 + i of
    // tile cc, row l16).
#pragma unroll 1
    for (int hh = 0; hh < 2; ++hh) {
      float4_t s[2];
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        float4_t acc = {0.f, 0.f, 0.f, 0.f};
        const int kbase = (32 * hh + 16 * jj + l16) * kKStride + 8 * g4;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const half8_t ah = *reinterpret_cast<const half8_t*>(khi + kbase + 32 * ks);
          const half8_t al = *reinterpret_cast<const half8_t*>(klo + kbase + 32 * ks);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, qh[ks], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(al, qh[ks], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, qlo[ks * 64], acc, 0, 0, 0);
        }
        s[jj] = acc;
      }
      float mx = kNegInf;
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tok = t0 + 32 * hh + 16 * jj + 4 * g4 + i;
          s[jj][i] = tok > pos ? kNegInf : s[jj][i];
          mx = fmaxf(mx, s[jj][i]);
        }
      mx = max4g(mx);
      // m_run stays -inf only while every token so far is masked (tokens past pos)
      const float mn = fmaxf(m_run, mx);
      const float corr = m_run == kNegInf ? 0.f : exp2f(m_run - mn);
      const float mref = mn == kNegInf ? 0.f : mn;
      m_run = mn;
      float ps = 0.f;
      half8_t pb;  // B operand of O^T = V^T P^T: tokens {4 g4 + i, 16 + 4 g4 + i} of the half
      {
        const uint2 va = *reinterpret_cast<const uint2*>(vnrm + 32 * hh + 4 * g4);
        const uint2 vb = *reinterpret_cast<const uint2*>(vnrm + 32 * hh + 16 + 4 * g4);
        const uint32_t vr[4] = {va.x, va.y, vb.x, vb.y};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float p = exp2f(s[e >> 2][e & 3] - mref);
          ps += p;
          const uint16_t nb = static_cast<uint16_t>(vr[e >> 1] >> (16 * (e & 1)));
          pb[e] = static_cast<_Float16>(p * h2f(nb));
        }
      }
      l_run = l_run * corr + ps;
      if (corr != 1.f) {
#pragma unroll
        for (int cc = 0; cc < 8; ++cc) o[cc] *= corr;
      }
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) {
        const _Float16* vrow = vh + (16 * cc + l16) * kVStride + 32 * hh + 4 * g4;
        const uint2 a0 = *reinterpret_cast<const uint2*>(vrow);
        const uint2 a1 = *reinterpret_cast<const uint2*>(vrow + 16);
        const uint4 u = make_uint4(a0.x, a0.y, a1.x, a1.y);
        o[cc] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, u), pb, o[cc], 0, 0, 0);
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
    for (int i = tid; i < kHeadDim * kHeadDim / 4; i += kAttnThreads) reinterpret_cast<float4*>(rv)[i] = src[i];
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
