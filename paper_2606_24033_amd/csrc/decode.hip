// Split pass of the packed-cache decode attention for gfx950 (Sec. 4: fused
// unpack -> codebook -> norm rescale -> QK and PV products -> online softmax,
// split along the key axis).
//
// Work mapping.  One workgroup = 8 waves = one (split, KV head, sequence[,
// layer]).  A wave owns 64-token tiles (two value tiles).  Both products run
// on 4x4x4 f16 MFMA blocks (16 independent 4x4 blocks per instruction):
//  * QK: block b holds tokens 4b..4b+3 of the tile, so lane l = 4b+i decodes
//    the key row of token l, 4 coordinates per step.  Every lane decodes the
//    same 4 stream positions in a step, so all lanes share one code width (no
//    divergence) and a step never mixes two groups.  The B operand is the
//    rotated query (4 coordinates x 4 heads), the same in every block.
//    A group's partial dot products are scaled by its fp16 radius in fp32.
//  * PV: block b holds output dims 4b..4b+3 (two instructions per 128 dims),
//    the contraction runs over 4 tokens per step.  Lane l = 4b+j decodes 4
//    tokens of dim (64h + l) straight from the value tile (codes of one
//    coordinate are contiguous there).
// Dequantization goes through lookup tables in LDS, replicated per lane so
// that random indices never collide on a bank: 4 codes per lookup for b <= 2
// (a 64-bit entry of four fp16 centroids), 2 codes for b = 3, 1 code above.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "layout.h"

namespace bgtq {
namespace {

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr float kNegInf = -__builtin_huge_valf();

// LDS map (bytes)
constexpr int kLut1 = 0;                        // b=1: 16 entries x 16 replicas x 8 B
constexpr int kLut2 = kLut1 + 16 * 16 * 8;      // b=2: 256 x 16 x 8
constexpr int kLut3 = kLut2 + 256 * 16 * 8;     // b=3: 64 (2 codes) x 32 x 4
constexpr int kLut4 = kLut3 + 64 * 32 * 4;      // b=4: 16 x 32 x 4 (fp16 in the low half)
constexpr int kLut5 = kLut4 + 16 * 32 * 4;      // b=5: 32 x 32 x 4
constexpr int kLutF = kLut5 + 32 * 32 * 4;      // b=6,7,8: plain fp16 tables at +0, +128, +384
constexpr int kQbuf = kLutF + 1024;             // rotated query per step: [step][set][hi,lo][head][4] fp16
constexpr int kPbuf = kQbuf + kMaxSteps * 2 * 2 * 4 * 8;  // per wave: [set][head][64 tokens] fp16
constexpr int kLdsBytes = kPbuf + kWaves * 1024;
static_assert(kLdsBytes <= 65536, "LDS budget");

__device__ __forceinline__ uint32_t lds32(const uint8_t* s, uint32_t off) {
  return *reinterpret_cast<const uint32_t*>(s + off);
}
__device__ __forceinline__ uint2 lds64(const uint8_t* s, uint32_t off) {
  return *reinterpret_cast<const uint2*>(s + off);
}
__device__ __forceinline__ half4_t as_half4(uint32_t lo, uint32_t hi) {
  uint2 u = make_uint2(lo, hi);
  return __builtin_bit_cast(half4_t, u);
}
__device__ __forceinline__ float h2f(uint32_t bits16) {
  return __half2float(__ushort_as_half(static_cast<unsigned short>(bits16)));
}

// Single-code table lookup for b >= 4 (returns the fp16 bits).
__device__ __forceinline__ uint32_t lut_one(const uint8_t* s, int b, uint32_t code, uint32_t rep32) {
  if (b == 4) return lds32(s, kLut4 + code * 128 + rep32) & 0xFFFFu;
  if (b == 5) return lds32(s, kLut5 + code * 128 + rep32) & 0xFFFFu;
  const uint32_t base = kLutF + (b == 6 ? 0 : (b == 7 ? 128 : 384));
  return *reinterpret_cast<const uint16_t*>(s + base + code * 2);
}

// Four consecutive b-bit codes at bit 0 of x -> four fp16 centroids.
__device__ __forceinline__ half4_t decode4(const uint8_t* s, uint32_t x, int b, uint32_t rep16,
                                           uint32_t rep32) {
  if (b <= 2) {
    const uint32_t e = x & ((1u << (4 * b)) - 1u);
    const uint2 u = lds64(s, (b == 1 ? kLut1 : kLut2) + e * 128 + rep16);
    return as_half4(u.x, u.y);
  }
  if (b == 3) {
    const uint32_t u0 = lds32(s, kLut3 + (x & 63u) * 128 + rep32);
    const uint32_t u1 = lds32(s, kLut3 + ((x >> 6) & 63u) * 128 + rep32);
    return as_half4(u0, u1);
  }
  const uint32_t m = (1u << b) - 1u;
  const uint32_t c0 = lut_one(s, b, x & m, rep32), c1 = lut_one(s, b, (x >> b) & m, rep32);
  const uint32_t c2 = lut_one(s, b, (x >> (2 * b)) & m, rep32);
  const uint32_t c3 = lut_one(s, b, b == 8 ? (x >> 24) : ((x >> (3 * b)) & m), rep32);
  return as_half4(c0 | (c1 << 16), c2 | (c3 << 16));
}

__device__ __forceinline__ float xmax4(float v) {
  v = fmaxf(v, __shfl_xor(v, 4, 64));
  v = fmaxf(v, __shfl_xor(v, 8, 64));
  v = fmaxf(v, __shfl_xor(v, 16, 64));
  return fmaxf(v, __shfl_xor(v, 32, 64));
}
__device__ __forceinline__ float xsum4(float v) {
  v += __shfl_xor(v, 4, 64);
  v += __shfl_xor(v, 8, 64);
  v += __shfl_xor(v, 16, 64);
  return v + __shfl_xor(v, 32, 64);
}
// value of lane (lane & ~3) | r
__device__ __forceinline__ float quad_get(float v, int r) {
  return __shfl(v, (static_cast<int>(threadIdx.x & 63) & ~3) | r, 64);
}

// PV for one 64-token tile with value width BV known at compile time: loads
// the lane's value words (dim 64h + lane of both value tiles) and runs the 16
// 4-token steps.  pw holds the wave's fp16 probabilities [set][head][token].
template <int NSET, int BV>
__device__ __forceinline__ void pv_tile(const uint8_t* smem, const uint8_t* pw, const uint32_t* __restrict__ vbase,
                                        int tiles_left, int lane, int jq, uint32_t rep16, uint32_t rep32,
                                        float4_t (&O)[NSET][2]) {
  uint32_t vw[4][BV + 1];
#pragma unroll
  for (int th = 0; th < 4; ++th) {
    const int tau = th >> 1, h = th & 1;
#pragma unroll
    for (int w = 0; w <= BV; ++w) vw[th][w] = 0;
    if (tau < tiles_left) {
      const uint32_t* src = vbase + (static_cast<size_t>(tau) * kHeadDim + 64 * h + lane) * BV;
      if constexpr (BV % 4 == 0) {
#pragma unroll
        for (int w = 0; w < BV; w += 4) {
          const uint4 v4 = *reinterpret_cast<const uint4*>(src + w);
          vw[th][w] = v4.x; vw[th][w + 1] = v4.y; vw[th][w + 2] = v4.z; vw[th][w + 3] = v4.w;
        }
      } else if constexpr (BV % 2 == 0) {
#pragma unroll
        for (int w = 0; w < BV; w += 2) {
          const uint2 v2 = *reinterpret_cast<const uint2*>(src + w);
          vw[th][w] = v2.x; vw[th][w + 1] = v2.y;
        }
      } else {
#pragma unroll
        for (int w = 0; w < BV; ++w) vw[th][w] = src[w];
      }
    }
  }
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int tau = k >> 3, sp = k & 7;
    constexpr int kBits = 4 * BV;
    const int vo = kBits * sp, w = vo >> 5, sh = vo & 31;
    half4_t ap[NSET];
#pragma unroll
    for (int s = 0; s < NSET; ++s) {
      const uint2 u = lds64(pw, ((s * 4 + jq) * 64 + 4 * k) * 2);
      ap[s] = as_half4(u.x, u.y);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t lo = vw[tau * 2 + h][w], hi = vw[tau * 2 + h][w + 1];
      const uint32_t x = (sh + kBits <= 32) ? (lo >> sh) : __builtin_amdgcn_alignbit(hi, lo, sh);
      const half4_t bvv = decode4(smem, x, BV, rep16, rep32);
#pragma unroll
      for (int s = 0; s < NSET; ++s) O[s][h] = __builtin_amdgcn_mfma_f32_4x4x4f16(ap[s], bvv, O[s][h], 0, 0, 0);
    }
  }
}

template <int NSET, int KWB>
__global__ __launch_bounds__(kThreads) void k_split_mfma(Dims d, const uint8_t* __restrict__ blob,
                                                         const int32_t* __restrict__ ctx_len, CachePtrs c,
                                                         const float* __restrict__ qp, float* __restrict__ part,
                                                         int n_splits, int split_len) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bq = lane >> 2, jq = lane & 3;
  const int split = blockIdx.x, kvh = blockIdx.y, lz = blockIdx.z;
  const int layer = d.layer >= 0 ? d.layer : lz / d.batch;
  const int seq = lz % d.batch;
  const int G = d.group, hqn = d.n_kv * G;
  const int cap = d.capacity, kw = d.k_words, bv = d.v_bits;
  const RowMeta* M = reinterpret_cast<const RowMeta*>(blob + kOffRows) + (layer * d.n_kv + kvh);
  const uint16_t* c16 = reinterpret_cast<const uint16_t*>(blob + kOffC16);
  const int n_steps = M->n_steps;

  // ---- lookup tables
  for (int i = tid; i < 16 * 16; i += kThreads) {
    const int e = i >> 4;
    const uint16_t* cb = c16 + cb_index(1);
    uint2 u = make_uint2(cb[e & 1] | (static_cast<uint32_t>(cb[(e >> 1) & 1]) << 16),
                         cb[(e >> 2) & 1] | (static_cast<uint32_t>(cb[(e >> 3) & 1]) << 16));
    *reinterpret_cast<uint2*>(smem + kLut1 + i * 8) = u;
  }
  for (int i = tid; i < 256 * 16; i += kThreads) {
    const int e = i >> 4;
    const uint16_t* cb = c16 + cb_index(2);
    uint2 u = make_uint2(cb[e & 3] | (static_cast<uint32_t>(cb[(e >> 2) & 3]) << 16),
                         cb[(e >> 4) & 3] | (static_cast<uint32_t>(cb[(e >> 6) & 3]) << 16));
    *reinterpret_cast<uint2*>(smem + kLut2 + i * 8) = u;
  }
  for (int i = tid; i < 64 * 32; i += kThreads) {
    const int e = i >> 5;
    const uint16_t* cb = c16 + cb_index(3);
    *reinterpret_cast<uint32_t*>(smem + kLut3 + i * 4) = cb[e & 7] | (static_cast<uint32_t>(cb[(e >> 3) & 7]) << 16);
  }
  for (int i = tid; i < 16 * 32; i += kThreads)
    *reinterpret_cast<uint32_t*>(smem + kLut4 + i * 4) = c16[cb_index(4) + (i >> 5)];
  for (int i = tid; i < 32 * 32; i += kThreads)
    *reinterpret_cast<uint32_t*>(smem + kLut5 + i * 4) = c16[cb_index(5) + (i >> 5)];
  for (int i = tid; i < 64 + 128 + 256; i += kThreads) {
    const int b = i < 64 ? 6 : (i < 192 ? 7 : 8);
    const int k = i < 64 ? i : (i < 192 ? i - 64 : i - 192);
    *reinterpret_cast<uint16_t*>(smem + kLutF + i * 2) = c16[cb_index(b) + k];
  }
  // ---- rotated queries as MFMA operands, one 4-coordinate slice per step.
  // fp16 alone would put ~2^-12 relative error on every logit term, so each
  // value is split into hi = fp16(q) and lo = fp16(q - hi) and both products
  // are accumulated in fp32.
  const float* qbase = qp + (static_cast<size_t>(lz) * hqn + kvh * G) * kHeadDim;
  for (int i = tid; i < n_steps * NSET * 4 * 4; i += kThreads) {
    const int k = i & 3, j = (i >> 2) & 3, set = (i >> 4) % NSET, st_i = (i >> 4) / NSET;
    const uint32_t st = M->step[st_i];
    const int p0 = (st >> 19) & 127, valid = (st >> 26) & 7;
    const int q = set * 4 + j;
    float v = 0.f;
    if (q < G && k < valid) v = qbase[q * kHeadDim + p0 + k];
    const _Float16 hi = static_cast<_Float16>(v);
    const _Float16 lo = static_cast<_Float16>(v - static_cast<float>(hi));
    uint8_t* qs = smem + kQbuf + (((st_i * 2 + set) * 2) * 4 + j) * 8 + k * 2;
    *reinterpret_cast<_Float16*>(qs) = hi;
    *reinterpret_cast<_Float16*>(qs + 32) = lo;
  }
  __syncthreads();

  const int ctx = min(ctx_len[seq], cap);
  const int t_begin = split * split_len;
  const int t_end = min(t_begin + split_len, ctx);
  const size_t row = (static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + kvh;
  const int ng = M->n_groups;
  const uint32_t rep16 = (lane & 15) * 8, rep32 = (lane & 31) * 4;
  const float vscale = 0.08838834764831845f;  // 1/sqrt(128)
  uint8_t* pw = smem + kPbuf + wave * 1024;

  float m_run[NSET], l_run[NSET];
  float4_t O[NSET][2];
#pragma unroll
  for (int s = 0; s < NSET; ++s) {
    m_run[s] = kNegInf;
    l_run[s] = 0.f;
    O[s][0] = float4_t{0.f, 0.f, 0.f, 0.f};
    O[s][1] = float4_t{0.f, 0.f, 0.f, 0.f};
  }

  for (int t0 = t_begin + wave * 64; t0 < t_end; t0 += kWaves * 64) {
    // ---------------- loads
    uint32_t rw[KWB + 1];
#pragma unroll
    for (int i = 0; i <= KWB; ++i) rw[i] = 0;
    const int tk = t0 + lane;
    if (tk < cap) {
      const uint32_t* src = c.k_codes + (row * cap + tk) * kw;
      if ((kw & 3) == 0) {
#pragma unroll
        for (int i = 0; i < KWB; i += 4) {
          if (i < kw) {
            const uint4 v = *reinterpret_cast<const uint4*>(src + i);
            rw[i] = v.x; rw[i + 1] = v.y; rw[i + 2] = v.z; rw[i + 3] = v.w;
          }
        }
      } else {
#pragma unroll
        for (int i = 0; i < KWB; ++i)
          if (i < kw) rw[i] = src[i];
      }
    }
    const bool quad_in = t0 + 4 * bq < cap;
    uint32_t kn[2 * kMaxGroups];
#pragma unroll
    for (int g = 0; g < kMaxGroups; ++g) {
      kn[2 * g] = 0;
      kn[2 * g + 1] = 0;
      if (g < ng && quad_in) {
        const uint2 u = *reinterpret_cast<const uint2*>(c.k_norms + (row * kMaxGroups + g) * cap + t0 + 4 * bq);
        kn[2 * g] = u.x;
        kn[2 * g + 1] = u.y;
      }
    }
    const uint2 vn = quad_in ? *reinterpret_cast<const uint2*>(c.v_norms + row * cap + t0 + 4 * bq)
                             : make_uint2(0, 0);
    // ---------------- QK
    float4_t L[NSET], acc[NSET];
#pragma unroll
    for (int s = 0; s < NSET; ++s) {
      L[s] = float4_t{0.f, 0.f, 0.f, 0.f};
      acc[s] = float4_t{0.f, 0.f, 0.f, 0.f};
    }
    bool fresh = true;
    for (int w = 0; w < kw; ++w) {
      const uint32_t cur = rw[w], nxt = rw[w + 1];
      const int s_end = M->word_step[w + 1];
      for (int si = M->word_step[w]; si < s_end; ++si) {
        const uint32_t st = M->step[si];
        const int sh = static_cast<int>(st & 1023u) - 32 * w;
        const int b = (st >> 10) & 15;
        const uint32_t x = (sh + 4 * b <= 32) ? (cur >> sh) : __builtin_amdgcn_alignbit(nxt, cur, sh);
        const half4_t a = decode4(smem, x, b, rep16, rep32);
#pragma unroll
        for (int s = 0; s < NSET; ++s) {
          const uint2 qh = lds64(smem, kQbuf + (((si * 2 + s) * 2) * 4 + jq) * 8);
          const uint2 ql = lds64(smem, kQbuf + (((si * 2 + s) * 2 + 1) * 4 + jq) * 8);
          acc[s] = __builtin_amdgcn_mfma_f32_4x4x4f16(a, as_half4(qh.x, qh.y),
                                                      fresh ? float4_t{0.f, 0.f, 0.f, 0.f} : acc[s], 0, 0, 0);
          acc[s] = __builtin_amdgcn_mfma_f32_4x4x4f16(a, as_half4(ql.x, ql.y), acc[s], 0, 0, 0);
        }
        fresh = false;
        if ((st >> 17) & 1u) {
          const int gi = 2 * ((st >> 14) & 7);
          const uint32_t nx = kn[gi], ny = kn[gi + 1];
          const float n0 = h2f(nx & 0xFFFFu), n1 = h2f(nx >> 16), n2 = h2f(ny & 0xFFFFu), n3 = h2f(ny >> 16);
#pragma unroll
          for (int s = 0; s < NSET; ++s) {
            L[s][0] = fmaf(n0, acc[s][0], L[s][0]);
            L[s][1] = fmaf(n1, acc[s][1], L[s][1]);
            L[s][2] = fmaf(n2, acc[s][2], L[s][2]);
            L[s][3] = fmaf(n3, acc[s][3], L[s][3]);
          }
          fresh = true;
        }
      }
    }

    // ---------------- online softmax over this tile
    const float vn4[4] = {h2f(vn.x & 0xFFFFu) * vscale, h2f(vn.x >> 16) * vscale, h2f(vn.y & 0xFFFFu) * vscale,
                          h2f(vn.y >> 16) * vscale};
#pragma unroll
    for (int s = 0; s < NSET; ++s) {
      float mx = kNegInf;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (t0 + 4 * bq + r >= t_end) L[s][r] = kNegInf;
        mx = fmaxf(mx, L[s][r]);
      }
      mx = xmax4(mx);
      const float mn = fmaxf(m_run[s], mx);
      const float corr = m_run[s] == kNegInf ? 0.f : __expf(m_run[s] - mn);
      float ps = 0.f;
      uint32_t ph[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = __expf(L[s][r] - mn);
        ps += p;
        const float pv = (t0 + 4 * bq + r < t_end) ? p * vn4[r] : 0.f;
        ph[r] = __half_as_ushort(__float2half_rn(pv));
      }
      ps = xsum4(ps);
      l_run[s] = l_run[s] * corr + ps;
      m_run[s] = mn;
      *reinterpret_cast<uint2*>(pw + ((s * 4 + jq) * 64 + 4 * bq) * 2) =
          make_uint2(ph[0] | (ph[1] << 16), ph[2] | (ph[3] << 16));
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float cr = quad_get(corr, r);
        O[s][0][r] *= cr;
        O[s][1][r] *= cr;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // ---------------- PV: 16 steps of 4 tokens
    {
      const int T0 = t0 / kTile;
      const int tiles_left = cap / kTile - T0;
      const uint32_t* vbase = c.v_codes + (row * (cap / kTile) + T0) * kHeadDim * bv;
      switch (bv) {
        case 1: pv_tile<NSET, 1>(smem, pw, vbase, tiles_left, lane, jq, rep16, rep32, O); break;
        case 2: pv_tile<NSET, 2>(smem, pw, vbase, tiles_left, lane, jq, rep16, rep32, O); break;
        case 3: pv_tile<NSET, 3>(smem, pw, vbase, tiles_left, lane, jq, rep16, rep32, O); break;
        case 4: pv_tile<NSET, 4>(smem, pw, vbase, tiles_left, lane, jq, rep16, rep32, O); break;
        case 5: pv_tile<NSET, 5>(smem, pw, vbase, tiles_left, lane, jq, rep16, rep32, O); break;
        case 6: pv_tile<NSET, 6>(smem, pw, vbase, tiles_left, lane, jq, rep16, rep32, O); break;
        case 7: pv_tile<NSET, 7>(smem, pw, vbase, tiles_left, lane, jq, rep16, rep32, O); break;
        default: pv_tile<NSET, 8>(smem, pw, vbase, tiles_left, lane, jq, rep16, rep32, O); break;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // ---------------- merge the 8 waves of the workgroup
  __syncthreads();
  float* fm = reinterpret_cast<float*>(smem);            // [wave][8] max
  float* fl = fm + kWaves * 8;                           // [wave][8] sum
  float* fo = fl + kWaves * 8;                           // [wave][8][128] accumulators
#pragma unroll
  for (int s = 0; s < NSET; ++s) {
    if (bq == 0) {
      fm[wave * 8 + s * 4 + jq] = m_run[s];
      fl[wave * 8 + s * 4 + jq] = l_run[s];
    }
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) fo[(wave * 8 + s * 4 + r) * kHeadDim + 64 * h + lane] = O[s][h][r];
  }
  __syncthreads();
  for (int i = tid; i < G * kHeadDim; i += kThreads) {
    const int q = i >> 7, dd = i & 127;
    float mx = kNegInf;
    for (int w = 0; w < kWaves; ++w) mx = fmaxf(mx, fm[w * 8 + q]);
    float l = 0.f, a = 0.f;
    if (mx != kNegInf) {
      for (int w = 0; w < kWaves; ++w) {
        const float mw = fm[w * 8 + q];
        if (mw == kNegInf) continue;
        const float e = __expf(mw - mx);
        l = fmaf(fl[w * 8 + q], e, l);
        a = fmaf(fo[(w * 8 + q) * kHeadDim + dd], e, a);
      }
    }
    float* pb = part + ((static_cast<size_t>(lz) * hqn + kvh * G + q) * n_splits + split) * 130;
    pb[2 + dd] = a;
    if (dd == 0) {
      pb[0] = mx;
      pb[1] = l;
    }
  }
}

}  // namespace

template <int NSET, int KWB>
static void launch_kw(const Dims& d, dim3 grid, const uint8_t* blob, const int32_t* ctx_len, const CachePtrs& c,
                      const DecodeWs& ws, hipStream_t s) {
  hipLaunchKernelGGL((k_split_mfma<NSET, KWB>), grid, dim3(kThreads), 0, s, d, blob, ctx_len, c, ws.qp, ws.part,
                     ws.n_splits, ws.split_len);
}

template <int NSET>
static void launch_set(const Dims& d, dim3 grid, const uint8_t* blob, const int32_t* ctx_len, const CachePtrs& c,
                       const DecodeWs& ws, hipStream_t s) {
  if (d.k_words <= 8)
    launch_kw<NSET, 8>(d, grid, blob, ctx_len, c, ws, s);
  else if (d.k_words <= 16)
    launch_kw<NSET, 16>(d, grid, blob, ctx_len, c, ws, s);
  else
    launch_kw<NSET, 32>(d, grid, blob, ctx_len, c, ws, s);
}

hipError_t launch_split_mfma(const Dims& d, const void* layout, const int32_t* ctx_len, const CachePtrs& c,
                             const DecodeWs& ws, hipStream_t s) {
  dim3 grid(ws.n_splits, d.n_kv, d.batch * d.n_lc);
  const uint8_t* blob = static_cast<const uint8_t*>(layout);
  if (d.group <= 4)
    launch_set<1>(d, grid, blob, ctx_len, c, ws, s);
  else
    launch_set<2>(d, grid, blob, ctx_len, c, ws, s);
  return hipGetLastError();
}

}  // namespace bgtq
