// HIP kernels of the Block-GTQ packed-cache path for gfx950 (MI355X).
//
//  k_quantize      : TQ-MSE encode (Sec. 2.2) of appended K rows per same-rate
//                    group (end of Sec. 3.2) and of V rows, dense b-bit pack.
//  (the packed-cache decode lives in decode_impl.h)
//  k_merge         : exact log-sum-exp merge of the splits + inverse V rotation.
//  k_split_fp16    : the same decode over an fp16 cache (comparator).
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

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
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
// Quantize + pack + append.  One workgroup per (value tile touched, KV head,
// sequence[, layer]).  Tokens of the tile outside [write_pos, write_pos+n_new)
// keep their packed bits.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_quantize(Dims d, const uint8_t* __restrict__ blob,
                                                  const void* __restrict__ kin,
                                                  const void* __restrict__ vin, int n_new,
                                                  const int32_t* __restrict__ wpos, CachePtrs c) {
  __shared__ float xk[kTile][kHeadDim];
  __shared__ float xv[kTile][kHeadDim];
  __shared__ uint8_t ck[kTile][kHeadDim];
  __shared__ uint8_t cv[kTile][kHeadDim];
  __shared__ float thr[kThresholdEntries];
  __shared__ RowMeta meta;

  const int tid = threadIdx.x;
  const int lz = blockIdx.z;
  const int layer = d.layer >= 0 ? d.layer : lz / d.batch;
  const int seq = lz % d.batch;
  const int head = blockIdx.y;
  const int wp = wpos[seq];
  if (wp < 0) return;
  const int tile = wp / kTile + blockIdx.x;
  const int t_lo = max(tile * kTile, wp);
  const int t_hi = min(min(tile * kTile + kTile, wp + n_new), d.capacity);
  if (t_lo >= t_hi) return;

  const float* gthr = reinterpret_cast<const float*>(blob + kOffThr);
  const float* rotkt = reinterpret_cast<const float*>(blob + kOffRotKT);
  const float* rotvt = reinterpret_cast<const float*>(blob + kOffRotVT);
  const RowMeta* gmeta =
      reinterpret_cast<const RowMeta*>(blob + kOffRows) + (layer * d.n_kv + head);

  for (int i = tid; i < static_cast<int>(sizeof(RowMeta) / 4); i += 256)
    reinterpret_cast<uint32_t*>(&meta)[i] = reinterpret_cast<const uint32_t*>(gmeta)[i];
  for (int i = tid; i < kThresholdEntries; i += 256) thr[i] = gthr[i];
  const size_t row = (static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + head;
  for (int idx = tid; idx < kTile * kHeadDim; idx += 256) {
    const int s = idx >> 7, dd = idx & 127;
    const int t = tile * kTile + s;
    if (t >= t_lo && t < t_hi) {
      const size_t off =
          ((static_cast<size_t>(lz) * n_new + (t - wp)) * d.n_kv + head) * kHeadDim + dd;
      xk[s][dd] = ld_in(kin, off, d.in_dtype);
      xv[s][dd] = ld_in(vin, off, d.in_dtype);
    }
  }
  __syncthreads();

  const int wave = tid >> 6, lane = tid & 63;
  if (t_hi - t_lo <= 4) {
    // Few tokens (a decode-step append): all four waves work on one token at
    // a time.  Norms: wave w sums groups w, w+4 and wave 3 the value row, in
    // the same order as the per-wave path below; rotations: thread p < 128
    // takes key stream position p, thread 128 + j value coordinate j.  Same
    // arithmetic as the per-wave path, so the codes are the same.
    __shared__ float gnrm[kMaxGroups + 1];
    const int ng = meta.n_groups;
    for (int t = t_lo; t < t_hi; ++t) {
      const int s = t - tile * kTile;
      for (int g = wave; g < ng; g += 4) {
        const int dg = meta.g_dim[g], p0 = meta.g_pos[g];
        float ss = 0.f;
        for (int i = lane; i < dg; i += 64) {
          const float x = xk[s][meta.dim[p0 + i]];
          ss = fmaf(x, x, ss);
        }
        ss = wave_sum(ss);
        if (lane == 0) gnrm[g] = sqrtf(ss);
      }
      if (wave == 3) {
        float ss = 0.f;
        for (int i = lane; i < kHeadDim; i += 64) ss = fmaf(xv[s][i], xv[s][i], ss);
        ss = wave_sum(ss);
        if (lane == 0) gnrm[kMaxGroups] = sqrtf(ss);
      }
      __syncthreads();
      if (tid < kHeadDim) {
        const int p = tid, g = meta.grp[p];
        const int b = meta.g_bits[g], dg = meta.g_dim[g], p0 = meta.g_pos[g], j = p - p0;
        const float nrm = gnrm[g];
        const float scale = nrm > 0.f ? sqrtf(static_cast<float>(dg)) / nrm : 0.f;
        const float* rt = rotkt + rotk_index(dg);
        float acc = 0.f;
#pragma unroll 16
        for (int i = 0; i < dg; ++i) acc = fmaf(rt[i * dg + j], xk[s][meta.dim[p0 + i]], acc);
        ck[s][p] = static_cast<uint8_t>(scalar_code(thr + thr_index(b), b, acc * scale));
        if (j == 0) c.k_norms[row * kMaxGroups * d.capacity + t * ((ng + 1) & ~1) + g] = __half_as_ushort(__float2half_rn(nrm));
      } else {
        const int j = tid - kHeadDim, b = d.v_bits;
        const float nrm = gnrm[kMaxGroups];
        const float scale = nrm > 0.f ? sqrtf(static_cast<float>(kHeadDim)) / nrm : 0.f;
        float acc = 0.f;
#pragma unroll 16
        for (int i = 0; i < kHeadDim; ++i) acc = fmaf(rotvt[i * kHeadDim + j], xv[s][i], acc);
        cv[s][j] = static_cast<uint8_t>(scalar_code(thr + thr_index(b), b, acc * scale));
        if (j == 0) c.v_norms[row * d.capacity + t] = __half_as_ushort(__float2half_rn(nrm));
      }
      __syncthreads();
    }
  }
  for (int s = wave; s < kTile && t_hi - t_lo > 4; s += 4) {
    const int t = tile * kTile + s;
    if (t < t_lo || t >= t_hi) continue;
    for (int g = 0; g < meta.n_groups; ++g) {
      const int b = meta.g_bits[g], dg = meta.g_dim[g], p0 = meta.g_pos[g];
      float ss = 0.f;
      for (int i = lane; i < dg; i += 64) {
        const float x = xk[s][meta.dim[p0 + i]];
        ss = fmaf(x, x, ss);
      }
      ss = wave_sum(ss);
      const float nrm = sqrtf(ss);
      const float scale = nrm > 0.f ? sqrtf(static_cast<float>(dg)) / nrm : 0.f;
      const float* rt = rotkt + rotk_index(dg);
      for (int j = lane; j < dg; j += 64) {
        float acc = 0.f;
        for (int i = 0; i < dg; ++i) acc = fmaf(rt[i * dg + j], xk[s][meta.dim[p0 + i]], acc);
        ck[s][p0 + j] = static_cast<uint8_t>(scalar_code(thr + thr_index(b), b, acc * scale));
      }
      if (lane == 0)
        c.k_norms[row * kMaxGroups * d.capacity + t * ((meta.n_groups + 1) & ~1) + g] =
            __half_as_ushort(__float2half_rn(nrm));
    }
    {
      const int b = d.v_bits;
      float ss = 0.f;
      for (int i = lane; i < kHeadDim; i += 64) ss = fmaf(xv[s][i], xv[s][i], ss);
      ss = wave_sum(ss);
      const float nrm = sqrtf(ss);
      const float scale = nrm > 0.f ? sqrtf(static_cast<float>(kHeadDim)) / nrm : 0.f;
      for (int j = lane; j < kHeadDim; j += 64) {
        float acc = 0.f;
        for (int i = 0; i < kHeadDim; ++i) acc = fmaf(rotvt[i * kHeadDim + j], xv[s][i], acc);
        cv[s][j] = static_cast<uint8_t>(scalar_code(thr + thr_index(b), b, acc * scale));
      }
      if (lane == 0) c.v_norms[row * d.capacity + t] = __half_as_ushort(__float2half_rn(nrm));
    }
  }
  __syncthreads();

  // key rows: word w of a row collects every code whose bits meet [32w, 32w+32)
  const int kw = d.k_words;
  for (int idx = tid; idx < kTile * kw; idx += 256) {
    const int s = idx / kw, w = idx - s * kw;
    const int t = tile * kTile + s;
    if (t < t_lo || t >= t_hi) continue;
    uint32_t word = 0;
    for (int p = meta.word_first[w]; p < kHeadDim; ++p) {
      const int rel = static_cast<int>(meta.bitoff[p]) - 32 * w;
      if (rel >= 32) break;
      const uint32_t code = ck[s][p];
      word |= rel >= 0 ? (code << rel) : (code >> (-rel));
    }
    c.k_codes[(row * d.capacity + t) * kw + w] = word;
  }
  // value tile: word w of coordinate j holds slots whose bits meet [32w, 32w+32)
  const int bv = d.v_bits;
  const uint64_t fmask = (1ull << bv) - 1;
  for (int idx = tid; idx < kHeadDim * bv; idx += 256) {
    const int j = idx / bv, w = idx - j * bv;
    const size_t addr =
        ((row * (d.capacity / kTile) + tile) * kHeadDim + j) * static_cast<size_t>(bv) + w;
    uint32_t word = c.v_codes[addr];
    for (int s = 0; s < kTile; ++s) {
      const int t = tile * kTile + s;
      if (t < t_lo || t >= t_hi) continue;
      const int rel = s * bv - 32 * w;
      if (rel <= -bv || rel >= 32) continue;
      const uint64_t code = cv[s][j];
      uint32_t m, v;
      if (rel >= 0) {
        m = static_cast<uint32_t>(fmask << rel);
        v = static_cast<uint32_t>(code << rel);
      } else {
        m = static_cast<uint32_t>(fmask >> (-rel));
        v = static_cast<uint32_t>(code >> (-rel));
      }
      word = (word & ~m) | (v & m);
    }
    c.v_codes[addr] = word;
  }
}

// ---------------------------------------------------------------------------
// fp16 comparator: same split structure over an uncompressed fp16 cache.
// ---------------------------------------------------------------------------
template <int G>
__global__ __launch_bounds__(256) void k_split_fp16(Dims d, const void* __restrict__ q,
                                                    const int32_t* __restrict__ ctx_len,
                                                    const __half* __restrict__ k16,
                                                    const __half* __restrict__ v16,
                                                    float* __restrict__ part, int n_splits,
                                                    int split_len) {
  __shared__ float sq[G][kHeadDim];
  __shared__ float pt[G][256];
  __shared__ float red[2][G][4];
  __shared__ float xch[G][kHeadDim];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int split = blockIdx.x, kvh = blockIdx.y, lz = blockIdx.z;
  const int layer = d.layer >= 0 ? d.layer : lz / d.batch;
  const int seq = lz % d.batch;
  const int hqn = d.n_kv * G;
  const int cap = d.capacity;
  const float qscale = 1.0f / sqrtf(static_cast<float>(kHeadDim));
  for (int i = tid; i < G * kHeadDim; i += 256)
    sq[i >> 7][i & 127] =
        ld_in(q, (static_cast<size_t>(lz) * hqn + kvh * G + (i >> 7)) * kHeadDim + (i & 127), d.in_dtype) * qscale;
  __syncthreads();

  const int ctx = min(ctx_len[seq], cap);
  const int t0 = split * split_len;
  const int t1 = min(t0 + split_len, ctx);
  const size_t row = (static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + kvh;
  const __half* kb = k16 + row * cap * kHeadDim;
  const __half* vb = v16 + row * cap * kHeadDim;

  float m_run[G], l_run[G], acc[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m_run[h] = kNegInf;
    l_run[h] = 0.f;
    acc[h] = 0.f;
  }
  const int j = tid & 127, half = tid >> 7;
  for (int c0 = t0; c0 < t1; c0 += 256) {
    const int nrow = min(256, t1 - c0);
    const bool valid = tid < nrow;
    float lg[G];
    if (valid) {
#pragma unroll
      for (int h = 0; h < G; ++h) lg[h] = 0.f;
      const __half2* kr = reinterpret_cast<const __half2*>(kb + static_cast<size_t>(c0 + tid) * kHeadDim);
      for (int p2 = 0; p2 < kHeadDim / 2; ++p2) {
        const float2 kv = __half22float2(kr[p2]);
#pragma unroll
        for (int h = 0; h < G; ++h) lg[h] = fmaf(sq[h][2 * p2], kv.x, fmaf(sq[h][2 * p2 + 1], kv.y, lg[h]));
      }
    } else {
#pragma unroll
      for (int h = 0; h < G; ++h) lg[h] = kNegInf;
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mx = wave_max(lg[h]);
      if (lane == 0) red[0][h][wave] = mx;
    }
    __syncthreads();
    float corr[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mt = fmaxf(fmaxf(red[0][h][0], red[0][h][1]), fmaxf(red[0][h][2], red[0][h][3]));
      const float mn = fmaxf(m_run[h], mt);
      corr[h] = m_run[h] == kNegInf ? 0.f : __expf(m_run[h] - mn);
      const float p = valid ? __expf(lg[h] - mn) : 0.f;
      pt[h][tid] = p;
      const float ps = wave_sum(p);
      if (lane == 0) red[1][h][wave] = ps;
      m_run[h] = mn;
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h) {
      l_run[h] = l_run[h] * corr[h] + (red[1][h][0] + red[1][h][1] + red[1][h][2] + red[1][h][3]);
      acc[h] *= corr[h];
    }
    const int s_end = min(half * 128 + 128, nrow);
    for (int s = half * 128; s < s_end; ++s) {
      const float val = __half2float(vb[static_cast<size_t>(c0 + s) * kHeadDim + j]);
#pragma unroll
      for (int h = 0; h < G; ++h) acc[h] = fmaf(pt[h][s], val, acc[h]);
    }
    __syncthreads();
  }
  if (half == 1) {
#pragma unroll
    for (int h = 0; h < G; ++h) xch[h][j] = acc[h];
  }
  __syncthreads();
  if (half == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float* pb = part + ((static_cast<size_t>(lz) * hqn + kvh * G + h) * n_splits + split) * 130;
      pb[2 + j] = acc[h] + xch[h][j];
      if (j == 0) {
        pb[0] = m_run[h];
        pb[1] = l_run[h];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Exact LSE merge over splits, then out = Pi_V^T o_rot (if rotv != null).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(128) void k_merge(Dims d, const float* __restrict__ part, int n_splits,
                                               const float* __restrict__ rotv, float* __restrict__ out) {
  __shared__ float os[kHeadDim];
  const int tid = threadIdx.x;
  const int hq = blockIdx.x, seq = blockIdx.y, lc = blockIdx.z;
  const int hqn = d.n_kv * d.group;
  const size_t lz = static_cast<size_t>(lc) * d.batch + seq;
  const float* P = part + (lz * hqn + hq) * n_splits * 130;
  float mx = kNegInf;
  for (int s = 0; s < n_splits; ++s) mx = fmaxf(mx, P[s * 130]);
  float l = 0.f, a = 0.f;
  if (mx != kNegInf) {
    for (int s = 0; s < n_splits; ++s) {
      const float ms = P[s * 130];
      if (ms == kNegInf) continue;
      const float e = __expf(ms - mx);
      l = fmaf(P[s * 130 + 1], e, l);
      a = fmaf(P[s * 130 + 2 + tid], e, a);
    }
  }
  const float o = l > 0.f ? a / l : 0.f;
  float r = o;
  if (rotv != nullptr) {
    os[tid] = o;
    __syncthreads();
    r = 0.f;
    for (int jj = 0; jj < kHeadDim; ++jj) r = fmaf(rotv[jj * kHeadDim + tid], os[jj], r);
  }
  out[(lz * hqn + hq) * kHeadDim + tid] = r;
}

}  // namespace

hipError_t launch_quantize_append(const Dims& d, const void* layout, const void* k, const void* v,
                                  int n_new, const int32_t* write_pos, const CachePtrs& c,
                                  hipStream_t s) {
  if (n_new <= 0) return hipSuccess;
  dim3 grid((n_new + kTile - 1) / kTile + 1, d.n_kv, d.batch * d.n_lc);
  hipLaunchKernelGGL(k_quantize, grid, dim3(256), 0, s, d, static_cast<const uint8_t*>(layout), k,
                     v, n_new, write_pos, c);
  return hipGetLastError();
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

template <int G>
static void launch_split_fp16_g(const Dims& d, const void* q, const int32_t* ctx, const void* k16,
                                const void* v16, const DecodeWs& ws, hipStream_t s) {
  dim3 grid(ws.n_splits, d.n_kv, d.batch * d.n_lc);
  hipLaunchKernelGGL(k_split_fp16<G>, grid, dim3(256), 0, s, d, q, ctx,
                     static_cast<const __half*>(k16), static_cast<const __half*>(v16), ws.part,
                     ws.n_splits, ws.split_len);
}

hipError_t launch_decode_fp16(const Dims& d, const void* q, const int32_t* ctx_len, const void* k16,
                              const void* v16, float* out, const DecodeWs& ws, hipStream_t s) {
  switch (d.group) {
    case 1: launch_split_fp16_g<1>(d, q, ctx_len, k16, v16, ws, s); break;
    case 2: launch_split_fp16_g<2>(d, q, ctx_len, k16, v16, ws, s); break;
    case 3: launch_split_fp16_g<3>(d, q, ctx_len, k16, v16, ws, s); break;
    case 4: launch_split_fp16_g<4>(d, q, ctx_len, k16, v16, ws, s); break;
    case 5: launch_split_fp16_g<5>(d, q, ctx_len, k16, v16, ws, s); break;
    case 6: launch_split_fp16_g<6>(d, q, ctx_len, k16, v16, ws, s); break;
    case 7: launch_split_fp16_g<7>(d, q, ctx_len, k16, v16, ws, s); break;
    case 8: launch_split_fp16_g<8>(d, q, ctx_len, k16, v16, ws, s); break;
    default: return hipErrorInvalidValue;
  }
  const int hqn = d.n_kv * d.group;
  hipLaunchKernelGGL(k_merge, dim3(hqn, d.batch, d.n_lc), dim3(128), 0, s, d, ws.part, ws.n_splits,
                     static_cast<const float*>(nullptr), out);
  return hipGetLastError();
}

}  // namespace bgtq
