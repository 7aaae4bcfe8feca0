// Protected fp16 window beside the packed cache (the "protected" regime of
// the reasoning evaluation, Sec. 6 and its appendix): the first n_sink rows
// of a sequence (attention sink) and its last n_recent rows stay fp16, the
// rows in between are read from the packed cache.  During decode the cache is
// [ sink (fp16) | packed | recent (fp16) ].
//
// Two kernels:
//  * k_window_append: copies appended K/V rows into the window (fp16);
//  * k_window_attn: per (layer in call, sequence, KV head), the attention
//    partial of the G query heads over the window rows (base-2 logits as in
//    the packed decode, accumulator in the original V domain), which the
//    packed decode's merge folds in.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "layout.h"

namespace bgtq {
namespace {

constexpr int kWinThreads = 512;
constexpr int kWinChunk = 136;  // window rows staged per round trip
constexpr int kMaxWinRows = kMaxSink + kMaxRecent;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInfW = -__builtin_huge_valf();

__device__ __forceinline__ float ld_in(const void* p, size_t i, int dtype) {  // BGTQ_BF16 = 1
  if (dtype == 1) return __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(p)[i]) << 16);
  return reinterpret_cast<const float*>(p)[i];
}

__device__ __forceinline__ int win_slot(int t, int n_sink, int n_recent) {
  return t < n_sink ? t : n_sink + (t - n_sink) % n_recent;
}

// grid (n_new, n_kv, n_lc * batch), 128 threads (one per dim).  Row i of the
// call sits at position t = write_pos[seq] + i; it is kept if t < n_sink or
// if it is one of the call's last n_recent rows (so that no two rows of one
// call write the same recent slot).
__global__ __launch_bounds__(kHeadDim) void k_window_append(Dims d, const void* __restrict__ k,
                                                            const void* __restrict__ v, int n_new,
                                                            const int32_t* __restrict__ write_pos, int n_sink,
                                                            int n_recent, _Float16* __restrict__ win) {
  const int i = blockIdx.x, kvh = blockIdx.y, lz = blockIdx.z;
  const int seq = lz % d.batch;
  const int layer = d.layer >= 0 ? d.layer : lz / d.batch;
  const int t = write_pos[seq] + i;
  if (t < 0) return;  // a negative position writes nothing (as in the packed append)
  const bool sink = t < n_sink;
  const bool recent = !sink && n_recent > 0 && i >= n_new - n_recent;
  if (!sink && !recent) return;
  const int dd = threadIdx.x;
  const size_t src = ((static_cast<size_t>(lz) * n_new + i) * d.n_kv + kvh) * kHeadDim + dd;
  const size_t wcap = static_cast<size_t>(n_sink + n_recent);
  _Float16* base = win + ((static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + kvh) * 2 * wcap * kHeadDim;
  const size_t slot = static_cast<size_t>(win_slot(t, n_sink, n_recent)) * kHeadDim + dd;
  base[slot] = static_cast<_Float16>(ld_in(k, src, d.in_dtype));
  base[wcap * kHeadDim + slot] = static_cast<_Float16>(ld_in(v, src, d.in_dtype));
}

// grid (n_kv, n_lc * batch), 512 threads.  Rows of the window at context T:
// n_s = min(n_sink, T) sink rows and n_r = min(n_recent, T - n_s) recent rows
// T - n_r .. T - 1 (the packed decode covers the rows in between).
__global__ __launch_bounds__(kWinThreads) void k_window_attn(Dims d, const void* __restrict__ q,
                                                             const int32_t* __restrict__ ctx_len,
                                                             const _Float16* __restrict__ win, int n_sink,
                                                             int n_recent, float* __restrict__ wpart) {
  __shared__ float qs[8][kHeadDim];
  __shared__ float sc[8][kMaxWinRows];
  __shared__ float ml[8][2];
  __shared__ float red[kWinThreads / 64][8][kHeadDim];
  __shared__ int slot_of[kMaxWinRows];
  __shared__ uint4 kst[kWinChunk * 16];  // staged key rows (fp16)
  __shared__ uint4 vst[kWinChunk * 16];  // staged value rows (fp16)
  const int kvh = blockIdx.x, lz = blockIdx.y;
  const int seq = lz % d.batch;
  const int layer = d.layer >= 0 ? d.layer : lz / d.batch;
  const int G = d.group, hqn = d.n_kv * G, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = min(ctx_len[seq], d.capacity);
  const int ns = min(n_sink, T), nr = min(n_recent, T - ns), W = ns + nr;
  const size_t wcap = static_cast<size_t>(n_sink + n_recent);
  const _Float16* kb = win + ((static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + kvh) * 2 * wcap * kHeadDim;
  const _Float16* vb = kb + wcap * kHeadDim;
  float* wp = wpart + (static_cast<size_t>(lz) * hqn + kvh * G) * 130;

  for (int i = tid; i < G * kHeadDim; i += kWinThreads)
    qs[i >> 7][i & 127] = ld_in(q, (static_cast<size_t>(lz) * hqn + kvh * G) * kHeadDim + i, d.in_dtype) *
                          (kLog2e * 0.08838834764831845f);  // log2 e / sqrt(d_h)
  for (int j = tid; j < W; j += kWinThreads) slot_of[j] = win_slot(j < ns ? j : T - nr + (j - ns), n_sink, n_recent);
  __syncthreads();

  // Window rows are staged through LDS in chunks of kWinChunk rows, 16 bytes
  // per thread and load, so that a chunk costs one memory round trip; the
  // first value chunk is loaded together with the first key chunk (the
  // paper's 4 + 128 window is one chunk: one round trip in all).
  const auto stage = [&](uint4* dst, const _Float16* src, int j0, int n) {
    for (int i = tid; i < n * 16; i += kWinThreads)
      dst[i] = reinterpret_cast<const uint4*>(src + static_cast<size_t>(slot_of[j0 + (i >> 4)]) * kHeadDim)[i & 15];
  };
  for (int j0 = 0; j0 < W; j0 += kWinChunk) {
    const int n = min(kWinChunk, W - j0);
    stage(kst, kb, j0, n);
    if (j0 == 0) stage(vst, vb, 0, n);
    __syncthreads();
    // logits: one (window row, head) pair per thread
    for (int i = tid; i < n * G; i += kWinThreads) {
      const int j = i / G, g = i - j * G;
      float s = 0.f;
#pragma unroll 4
      for (int c = 0; c < kHeadDim / 8; ++c) {
        const uint4 w = kst[j * 16 + c];
        const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const _Float16 lo = __builtin_bit_cast(_Float16, static_cast<uint16_t>(u[h] & 0xFFFFu));
          const _Float16 hi = __builtin_bit_cast(_Float16, static_cast<uint16_t>(u[h] >> 16));
          s = fmaf(qs[g][8 * c + 2 * h], static_cast<float>(lo), s);
          s = fmaf(qs[g][8 * c + 2 * h + 1], static_cast<float>(hi), s);
        }
      }
      sc[g][j0 + j] = s;
    }
    __syncthreads();
  }

  // softmax per head: one wave per head
  for (int g = wave; g < G; g += kWinThreads / 64) {
    float m = kNegInfW;
    for (int j = lane; j < W; j += 64) m = fmaxf(m, sc[g][j]);
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    float l = 0.f;
    if (m != kNegInfW) {
      for (int j = lane; j < W; j += 64) {
        const float p = exp2f(sc[g][j] - m);
        sc[g][j] = p;
        l += p;
      }
    }
    for (int o = 32; o > 0; o >>= 1) l += __shfl_xor(l, o);
    if (lane == 0) {
      ml[g][0] = m;
      ml[g][1] = l;
    }
  }
  __syncthreads();

  // sum_j p_j v_j in the original V domain (the packed decode adds it after
  // its output rotation): lane = a pair of dims, wave w takes the rows
  // j = w mod (waves) of each staged value chunk, then the waves' sums are
  // added through LDS
  float2 acc[8];
#pragma unroll
  for (int g = 0; g < 8; ++g) acc[g] = make_float2(0.f, 0.f);
  for (int j0 = 0; j0 < W; j0 += kWinChunk) {
    const int n = min(kWinChunk, W - j0);
    if (j0 > 0) {
      __syncthreads();  // the previous chunk is consumed
      stage(vst, vb, j0, n);
      __syncthreads();
    }
    const uint32_t* vrow = reinterpret_cast<const uint32_t*>(vst);
    for (int j = wave; j < n; j += kWinThreads / 64) {
      const uint32_t vv = vrow[j * (kHeadDim / 2) + lane];
      const float v0 = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(vv & 0xFFFFu)));
      const float v1 = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(vv >> 16)));
#pragma unroll
      for (int g = 0; g < 8; ++g)
        if (g < G) {
          acc[g].x = fmaf(sc[g][j0 + j], v0, acc[g].x);
          acc[g].y = fmaf(sc[g][j0 + j], v1, acc[g].y);
        }
    }
  }
#pragma unroll
  for (int g = 0; g < 8; ++g)
    if (g < G) {
      red[wave][g][2 * lane] = acc[g].x;
      red[wave][g][2 * lane + 1] = acc[g].y;
    }
  __syncthreads();
  for (int i = tid; i < G * kHeadDim; i += kWinThreads) {
    const int g = i >> 7, dd = i & 127;
    float a = 0.f;
#pragma unroll
    for (int w = 0; w < kWinThreads / 64; ++w) a += red[w][g][dd];
    wp[g * 130 + 2 + dd] = a;
    if (dd == 0) {
      wp[g * 130] = ml[g][0];
      wp[g * 130 + 1] = ml[g][1];
    }
  }
}

}  // namespace

hipError_t launch_window_append(const Dims& d, const void* k, const void* v, int n_new, const int32_t* write_pos,
                                int n_sink, int n_recent, _Float16* window, hipStream_t s) {
  dim3 grid(n_new, d.n_kv, d.n_lc * d.batch);
  hipLaunchKernelGGL(k_window_append, grid, dim3(kHeadDim), 0, s, d, k, v, n_new, write_pos, n_sink, n_recent,
                     window);
  return hipGetLastError();
}

hipError_t launch_window_attn(const Dims& d, const void* q, const int32_t* ctx_len, const _Float16* window,
                              int n_sink, int n_recent, float* wpart, hipStream_t s) {
  dim3 grid(d.n_kv, d.n_lc * d.batch);
  hipLaunchKernelGGL(k_window_attn, grid, dim3(kWinThreads), 0, s, d, q, ctx_len, window, n_sink, n_recent, wpart);
  return hipGetLastError();
}

}  // namespace bgtq
