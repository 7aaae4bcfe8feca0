// Launchers of the HIP kernels (internal; the public surface is blockgtq.h).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bgtq {

struct Dims {
  int n_layers, batch, n_kv, group, capacity, k_words, v_bits, in_dtype;
  int layer;      // >= 0: one layer; -1: all layers
  int n_lc;       // layers in this call (1 or n_layers)
  int max_ctx;    // decode calls: the host's bound on ctx_len (outputs of a sequence outside [0, max_ctx] are NaN)
};

struct CachePtrs {
  uint32_t* k_codes;
  uint16_t* k_norms;
  uint32_t* v_codes;
  uint16_t* v_norms;
};

hipError_t launch_quantize_append(const Dims& d, const void* layout, const void* k,
                                  const void* v, int n_new, const int32_t* write_pos,
                                  const CachePtrs& c, hipStream_t s);
// The same for appends of more than a few rows (quantize.hip, fp32 MFMAs):
// k and v 16-byte aligned.
hipError_t launch_quantize_prefill(const Dims& d, const void* layout, const void* k, const void* v, int n_new,
                                   const int32_t* write_pos, const CachePtrs& c, hipStream_t s);

// Workspace carve-up of one decode call.
struct DecodeWs {
  int32_t* counters;  // [n_lc][batch][n_kv] finished-split counters (zero between calls)
  float* part;        // [n_lc][batch][Hq][n_splits][130] (m, l, acc[128])
  int n_splits;       // splits actually launched
  int split_len;      // tokens per split, multiple of 64
  // Protected fp16 window (null part: none).  The packed pass then covers
  // rows [n_s, T - n_r) of a context of T rows, n_s = min(n_sink, T),
  // n_r = min(n_recent, T - n_s), and the merge adds the window's partial
  // [n_lc][batch][Hq][130] (m, l, acc[128] in the original V domain).
  const float* wpart = nullptr;
  int n_sink = 0, n_recent = 0;
};

// Window sizes: the sink must end inside the first 64-row tile (the packed
// pass masks rows below it there only).
constexpr int kMaxSink = 63;
constexpr int kMaxRecent = 1024;

// Pre-RoPE decode-step inputs -> RoPE'd fp32 q, k and fp32 v (same layouts
// as the decode / append inputs of one row), and ctx[b] = pos[b] + 1.
hipError_t launch_rope_step(const Dims& d, double base, const void* q, const void* k, const void* v,
                            const int32_t* pos, float* qo, float* ko, float* vo, int32_t* ctx, hipStream_t s);

// Kernel-side view of the window arguments.
struct WinArgs {
  const float* part;
  int n_sink, n_recent;
};

// Protected window (a second fp16 store beside the packed cache): fp16
// [n_layers][batch][n_kv][2][n_sink + n_recent][128], keys then values;
// position t < n_sink sits in slot t, a later one in slot
// n_sink + (t - n_sink) mod n_recent.
hipError_t launch_window_append(const Dims& d, const void* k, const void* v, int n_new, const int32_t* write_pos,
                                int n_sink, int n_recent, _Float16* window, hipStream_t s);
// The window's attention partial of every (layer in call, sequence, query
// head), written to wpart for the packed decode's merge.
hipError_t launch_window_attn(const Dims& d, const void* q, const int32_t* ctx_len, const _Float16* window,
                              int n_sink, int n_recent, float* wpart, hipStream_t s);

// Packed decode (decode_impl.h), one entry per value code width
// (decode_bv1.hip .. decode_bv8.hip): query rotation, split pass and the
// merge of the splits in a single kernel.
#define BGTQ_DECL_SPLIT(N)                                                                                \
  hipError_t launch_split_bv##N(const Dims& d, const void* layout, const void* q, const int32_t* ctx_len, \
                                const CachePtrs& c, float* out, const DecodeWs& ws, hipStream_t s);
BGTQ_DECL_SPLIT(1)
BGTQ_DECL_SPLIT(2)
BGTQ_DECL_SPLIT(3)
BGTQ_DECL_SPLIT(4)
BGTQ_DECL_SPLIT(5)
BGTQ_DECL_SPLIT(6)
BGTQ_DECL_SPLIT(7)
BGTQ_DECL_SPLIT(8)
#undef BGTQ_DECL_SPLIT

hipError_t launch_decode_packed(const Dims& d, const void* layout, const void* q,
                                const int32_t* ctx_len, const CachePtrs& c, float* out,
                                const DecodeWs& ws, hipStream_t s);

hipError_t launch_decode_fp16(const Dims& d, const void* q, const int32_t* ctx_len,
                              const void* k16, const void* v16, float* out,
                              const DecodeWs& ws, hipStream_t s);

// Causal prefill attention over the packed cache of one layer (prefill.hip):
// the query rotation into qr_ws, then the attention into out.
hipError_t launch_prefill_attn(const Dims& d, const void* layout, const void* q, int n_q,
                               const int32_t* q_pos0, int max_pos, const CachePtrs& c, float* qr_ws,
                               float* out, hipStream_t s);

// Streaming read of `bytes` (a multiple of 16, 16-byte aligned) at src;
// writes sink[0] only in a case no real input reaches (probe.hip).
hipError_t launch_read_probe(const void* src, size_t bytes, uint32_t* sink, hipStream_t s);

// No-allocation decode (noalloc.hip): the current device's static scratch
// array (BGTQ_NOALLOC_SCRATCH_BYTES), its address looked up once per device;
// and a fill kernel that zeroes n split counters.
hipError_t noalloc_scratch(void** out);
hipError_t launch_clear_counters(int32_t* counters, int n, hipStream_t s);

}  // namespace bgtq
