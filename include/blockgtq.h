/*
 * blockgtq.h -- C ABI of the Block-GTQ packed-cache serving path on MI355X.
 *
 * Paper: "RoPE-Aware Bit Allocation for KV-Cache Quantization" (Block-GTQ).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Return value: 0 (BGTQ_OK) on success, a negative BGTQ_E* code on error.
 *    blockgtq_last_error() returns a message for the calling thread's last
 *    error.  No C++ exception crosses this boundary.  Argument errors are
 *    detected on the host before anything is enqueued.
 *  - Ownership: the caller owns every buffer.  The library never allocates
 *    device memory and keeps no state between calls; the device layout blob
 *    built by blockgtq_layout_init holds all constants.
 *  - Pointers named d_* and the cache / input / output pointers of the async
 *    calls are device pointers.  Host pointers are named h_* or documented so.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    The async calls only enqueue work; their device inputs must stay alive
 *    until the stream reaches them.  They neither allocate nor synchronise.
 *  - Shapes: head_dim d_h = 128 (L = 64 RoPE blocks); RoPE block i is the pair
 *    of dims (i, i + 64).  Group size G = query heads per KV head.
 *
 * Packed cache layout (per layer, sequence and KV head; all little-endian)
 * ---------------------------------------------------------------------
 *  k_codes : uint32 [n_layers][batch][n_kv_heads][capacity][k_words]
 *            One key row = the codes of every same-rate group, groups in
 *            ascending bit width, inside a group the rotated coordinates in
 *            order; each code is a dense b-bit field, LSB first; stream bit o
 *            is bit (o % 32) of word (o / 32).  k_words = ceil(2 B / 32).
 *  k_norms : fp16  [n_layers][batch][n_kv_heads][capacity * 8]
 *            Token-major radii: with n_g same-rate groups in the (layer, KV
 *            head) and S = n_g rounded up to even, token t's group radii sit
 *            at [t*S, t*S + n_g) in group ordinal (ascending b) order, so one
 *            4/8/12/16-byte load reads a token's radii.  Slots past n_g stay 0.
 *  v_codes : uint32 [n_layers][batch][n_kv_heads][capacity/32][d_h][b_v]
 *            Tiles of 32 tokens.  For rotated coordinate j the 32 codes of a
 *            tile form one 32*b_v-bit string; token slot s = t % 32 occupies
 *            bits [s*b_v, s*b_v + b_v).
 *  v_norms : fp16  [n_layers][batch][n_kv_heads][capacity]
 *  capacity must be a multiple of 64.  The caller zero-fills the cache once.
 */
#ifndef BLOCKGTQ_H
#define BLOCKGTQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  BGTQ_OK = 0,
  BGTQ_EINVAL = -1,       /* bad argument (shape, pointer, value)             */
  BGTQ_EBUDGET = -2,      /* bit budget outside [L*b_min, L*b_max]            */
  BGTQ_ECAPACITY = -3,    /* append or context beyond the cache capacity      */
  BGTQ_EWORKSPACE = -4,   /* workspace smaller than blockgtq_workspace_bytes  */
  BGTQ_EUNSUPPORTED = -5, /* configuration this build does not handle         */
  BGTQ_EHIP = -6          /* a HIP runtime call failed (message has details)  */
};

enum { BGTQ_FP32 = 0, BGTQ_BF16 = 1 };

/* Message for the calling thread's most recent error ("" if none). */
const char* blockgtq_last_error(void);

typedef struct {
  int32_t n_layers;    /* layers held by the cache                          */
  int32_t batch;       /* sequences                                         */
  int32_t n_kv_heads;  /* KV heads per layer                                */
  int32_t group;       /* query heads per KV head (G), 1..8                 */
  int32_t head_dim;    /* d_h; must be 128                                  */
  int32_t capacity;    /* rows per (layer, sequence, KV head); multiple of 64 */
  int32_t k_budget;    /* B = sum of the 64 block widths of a key head; the
                          K row holds 2B bits (K3 -> 192, K2 -> 128)         */
  int32_t v_bits;      /* b_V, 1..8                                         */
  int32_t in_dtype;    /* BGTQ_FP32 or BGTQ_BF16 for K, V and Q inputs       */
} bgtq_config;

typedef struct {
  void* k_codes; /* device, see layout above; each of the four buffers     */
  void* k_norms; /* 16-byte aligned (EINVAL otherwise: the kernels read    */
  void* v_codes; /* them with 16-byte loads)                               */
  void* v_norms;
} bgtq_cache;

/* ---- (a0) energy score -------------------------------------------------
 * Eq. (scoring-layer-head-energy) in Sec. 3.1, in its GQA form from the
 * calibration appendix: for each RoPE block i,
 *   s_i = 1/2 ( mean over tokens t and heads g of ||q_{g,t}^(i)||^2
 *               + mean over tokens t of ||k_t^(i)||^2 ).
 * Host, synchronous.  h_q: float [n_tokens][group][head_dim], h_k: float
 * [n_tokens][head_dim] (pre- or post-RoPE: block norms are RoPE-invariant).
 * h_scores_out: double [head_dim/2].  EINVAL on null pointers, n_tokens < 1,
 * group < 1 or odd head_dim. */
int blockgtq_energy_scores(const float* h_q, const float* h_k, int32_t n_tokens,
                           int32_t group, int32_t head_dim, double* h_scores_out);

/* ---- (a1) greedy allocator ---------------------------------------------
 * Algorithm 1 (Sec. 3.2): minimise J(b) = sum_i s_i 4^-b_i subject to
 * b_min <= b_i <= b_max and sum_i b_i = budget, by handing out bits one at a
 * time to the block with the largest marginal gain (3/4) s_i 4^-b_i.
 * Equal gains go to the lowest block index.  Host, synchronous, pure.
 * h_scores: double [n_rows][n_blocks], each finite and >= 0 (else EINVAL).
 * budget in [n_blocks*b_min, n_blocks*b_max] (else EBUDGET);
 * 1 <= b_min <= b_max <= 8.  h_bits_out: uint8 [n_rows][n_blocks]. */
int blockgtq_allocate(const double* h_scores, int32_t n_rows, int32_t n_blocks,
                      int32_t budget, int32_t b_min, int32_t b_max, uint8_t* h_bits_out);

/* ---- codebook ----------------------------------------------------------
 * The scalar quantizer of TQ-MSE (Sec. 2.2) at b bits: Gaussian Lloyd-Max
 * centroids rounded to fp16, and the 2^b - 1 decision thresholds (midpoints
 * of adjacent fp16 centroids, exact in fp32).  Host, synchronous.
 * h_c16_out: uint16 fp16 bit patterns [2^b]; h_thr_out: float [2^b - 1]
 * (either may be NULL).  EINVAL unless 1 <= b <= 8. */
int blockgtq_codebook(int32_t b, uint16_t* h_c16_out, float* h_thr_out);

/* ---- sizing ------------------------------------------------------------ */
int blockgtq_layout_bytes(const bgtq_config* cfg, size_t* bytes_out);
int blockgtq_cache_bytes(const bgtq_config* cfg, size_t* k_codes, size_t* k_norms,
                         size_t* v_codes, size_t* v_norms);
/* Workspace of one blockgtq_decode_attn (or _fp16) call: n_layers_in_call =
 * 1 for a single layer, cfg->n_layers for layer = -1.  n_splits as passed to
 * the call (0 = the heuristic for max_ctx).  The workspace starts with one int32
 * counter per (layer in call, sequence, KV head) that the kernel uses to find
 * the last split to finish: it must be zero-filled once before its first
 * use, and every completed call leaves it zero again.  Calls that share a
 * workspace must not overlap in time (one stream, or ordered by events). */
int blockgtq_workspace_bytes(const bgtq_config* cfg, int32_t n_layers_in_call,
                             int32_t n_splits, int32_t max_ctx, size_t* bytes_out);

/* ---- (a2) layout build --------------------------------------------------
 * Same-rate grouping (end of Sec. 3.2) and the static layout metadata that
 * the packed cache needs (Sec. 4): groups G_b = {i : b_i = b} in ascending
 * b, each block contributing dims (i, i+64); per-position widths and bit
 * offsets; the rotations and codebooks.  Uploads everything into the
 * caller's device buffer d_layout (blockgtq_layout_bytes bytes) and waits
 * for the copy (synchronous).
 * h_k_bits: uint8 [n_layers][n_kv_heads][64], each row summing to k_budget.
 * h_rot_k : float, the K rotations for d = 2, 4, ..., 128 concatenated, each
 *           d x d row-major (Pi maps a group vector x to Pi x); 357760 floats.
 * h_rot_v : float [128][128], row-major.
 * Rotations must be orthogonal (not checked beyond finiteness). */
int blockgtq_layout_init(const bgtq_config* cfg, const uint8_t* h_k_bits,
                         const float* h_rot_k, const float* h_rot_v, void* d_layout,
                         void* stream);

/* ---- (a3-a5) quantize + pack + append -----------------------------------
 * TQ-MSE (Sec. 2.2) per same-rate K group and per V row: n = ||x||,
 * z = sqrt(d) Pi x / n, code_j = #{thresholds <= z_j}, radius stored fp16;
 * codes packed into the cache layout above.  Async on `stream`.
 * layer in [0, n_layers) or -1 for all layers.
 * d_k, d_v: post-RoPE keys / values in cfg->in_dtype,
 *   [batch][n_new][n_kv_heads][head_dim]  (layer >= 0), or
 *   [n_layers][batch][n_new][n_kv_heads][head_dim]  (layer == -1);
 *   16-byte aligned (EINVAL otherwise).  Appends of up to 4 rows (decode
 *   steps) run one latency-oriented kernel; longer ones (prefill) one launch
 *   of key and value workgroups on fp32 MFMAs, a dense 128 x 128 product
 *   per row.
 * d_write_pos: int32 [batch]; sequence b's tokens go to rows
 *   d_write_pos[b] .. d_write_pos[b] + n_new - 1.  The caller guarantees
 *   d_write_pos[b] + n_new <= capacity (rows past capacity are not written)
 *   and advances its own lengths.  Calls touching the same rows must not
 *   overlap in time. */
int blockgtq_quantize_append(const bgtq_config* cfg, const void* d_layout, int32_t layer,
                             const void* d_k, const void* d_v, int32_t n_new,
                             const int32_t* d_write_pos, const bgtq_cache* cache,
                             void* stream);

/* ---- (a6-a8) split-context decode attention over the packed cache -------
 * Sec. 4: each query attends rows [0, d_ctx_len[b]) of its KV head with
 * logits q . k_hat / sqrt(d_h) and a softmax, the keys and values decoded
 * from the packed codes inside the kernel (no fp16 cache is written); the
 * context is split along the key axis into n_splits ranges whose partial
 * (max, sum, accumulator) states are merged exactly by log-sum-exp.  The
 * query is rotated into each group's code domain first (the Q-side rotation).
 * d_q: post-RoPE queries in cfg->in_dtype, [batch][n_kv_heads*group][head_dim]
 *      (layer >= 0) or [n_layers][batch][...][head_dim] (layer == -1);
 *      4-byte aligned (EINVAL otherwise).
 * d_ctx_len: int32 [batch], each in [0, max_ctx]; a sequence with 0 rows
 *      gets an all-zero output.  A length outside [0, max_ctx] (it is read on
 *      the device, so the call cannot reject it) makes that sequence's
 *      outputs NaN; no row is dropped silently and nothing outside the cache
 *      is read.
 * max_ctx: host-side upper bound of d_ctx_len (<= capacity), sizes the splits.
 * d_out: float, same shape as d_q.
 * d_workspace / ws_bytes: see blockgtq_workspace_bytes (EWORKSPACE if short;
 *      zero-filled before first use).  One kernel launch: the query rotation,
 *      the split pass and the merge of the splits.
 * n_splits: 0 = heuristic, else 1 .. 4096.  The (sequence, KV head, split)
 *      workgroups are dispatched in the layout's order of estimated row cost,
 *      most expensive first; the result does not depend on the order. */
int blockgtq_decode_attn(const bgtq_config* cfg, const void* d_layout, int32_t layer,
                         const void* d_q, const int32_t* d_ctx_len, int32_t max_ctx,
                         const bgtq_cache* cache, float* d_out, void* d_workspace,
                         size_t ws_bytes, int32_t n_splits, void* stream);

/* ---- fp16 comparator ----------------------------------------------------
 * The same split-context decode over an uncompressed fp16 cache, the
 * baseline the packed path's speedup is reported against (the paper compares
 * with fp16 FlashAttention-2 decode, Sec. 6 deployment).
 * d_k16, d_v16: fp16 [n_layers][batch][n_kv_heads][capacity][head_dim].
 * Other arguments as blockgtq_decode_attn (no layout blob: no codes, no
 * rotations); the same MFMA products, softmax and split merge. */
int blockgtq_decode_attn_fp16(const bgtq_config* cfg, int32_t layer, const void* d_q,
                              const int32_t* d_ctx_len, int32_t max_ctx,
                              const void* d_k16, const void* d_v16, float* d_out,
                              void* d_workspace, size_t ws_bytes, int32_t n_splits,
                              void* stream);

/* ---- (f1) prefill attention over the packed cache -----------------------
 * Causal attention of a prompt's queries over the packed cache of one layer
 * (Sec. 4, prefill paragraph): query i of sequence b sits at absolute position
 * d_q_pos0[b] + i and attends cache rows 0 .. that position, which must have
 * been appended before (blockgtq_quantize_append of the prompt's K/V).  Each
 * workgroup owns 256 query rows (position x head), decodes every packed key /
 * value tile of its range once into LDS for all of them, and runs QK^T and PV
 * on MFMAs under a causal mask and an online softmax; nothing fp16 is written
 * to HBM.  Async on `stream`; no allocation.
 * layer: 0 .. n_layers-1 (one layer per call).
 * d_q: post-RoPE [batch][n_q][n_kv_heads*group][128] in in_dtype, 4-byte
 *      aligned.  d_out: float, same shape.
 * d_q_pos0: device int32 [batch].  max_pos (host): an upper bound of every
 *      d_q_pos0[b] + n_q - 1, below capacity (ECAPACITY otherwise); positions
 *      are clamped into [0, max_pos] on the device, so every read stays
 *      inside the cache.
 * d_workspace / ws_bytes: blockgtq_prefill_workspace_bytes (the rotated
 *      queries, batch x n_q x n_kv_heads*group x 128 floats); any contents. */
int blockgtq_prefill_workspace_bytes(const bgtq_config* cfg, int32_t n_q, size_t* bytes_out);
int blockgtq_prefill_attn(const bgtq_config* cfg, const void* d_layout, int32_t layer,
                          const void* d_q, int32_t n_q, const int32_t* d_q_pos0, int32_t max_pos,
                          const bgtq_cache* cache, float* d_out, void* d_workspace,
                          size_t ws_bytes, void* stream);

/* ---- (f4) protected fp16 window ------------------------------------------
 * The "protected" regime of the reasoning evaluation (Sec. 6, AIME paragraph,
 * and the buffer configurations of its appendix): during decode the cache of
 * a sequence with T rows reads as [sink | packed | recent], where the first
 * n_s = min(n_sink, T) rows and the last n_r = min(n_recent, T - n_s) rows
 * are kept in fp16 and the rows in between come from the packed cache (the
 * paper's setting is n_sink = 4, n_recent = 128; 0 and 0 is the no-buffer
 * regime).  The packed cache still receives every row
 * (blockgtq_quantize_append); the window is a second, caller-owned store.
 *
 * d_window: fp16 [n_layers][batch][n_kv_heads][2][n_sink + n_recent][128],
 *   keys then values; position t < n_sink lives in slot t, a later position
 *   in slot n_sink + (t - n_sink) mod n_recent (a ring).
 * n_sink in 0..63 (the sink ends inside the first 64-row tile of the packed
 * pass), n_recent in 0..1024; EINVAL otherwise.  With both 0 the window is
 * empty and d_window may be NULL. */
int blockgtq_window_bytes(const bgtq_config* cfg, int32_t n_sink, int32_t n_recent, size_t* bytes_out);

/* Writes the fp16 copies of appended rows into the window (async on
 * `stream`).  Arguments as blockgtq_quantize_append (same d_k / d_v layouts
 * and positions); a row at position t is written if t < n_sink or if it is
 * one of the call's last n_recent rows, so a chunk longer than the recent
 * window leaves exactly its last n_recent rows in the ring.  Call it for
 * every row that blockgtq_quantize_append receives. */
int blockgtq_window_append(const bgtq_config* cfg, int32_t layer, const void* d_k, const void* d_v, int32_t n_new,
                           const int32_t* d_write_pos, int32_t n_sink, int32_t n_recent, void* d_window,
                           void* stream);

/* Workspace of blockgtq_decode_attn_protected: blockgtq_workspace_bytes plus
 * the window's partials ([n_layers_in_call][batch][n_kv_heads*group][130]
 * floats).  The counters at its start follow the same rules (zero-filled once
 * before first use; every completed call leaves them zero). */
int blockgtq_protected_workspace_bytes(const bgtq_config* cfg, int32_t n_layers_in_call, int32_t n_splits,
                                       int32_t max_ctx, size_t* bytes_out);

/* Decode attention over [sink | packed | recent]: arguments as
 * blockgtq_decode_attn, plus the window.  Two launches on `stream`: the
 * window kernel (exact fp32 logits and weights over the fp16 rows, its
 * partial written into the workspace), then the packed decode over rows
 * [n_s, T - n_r) whose merge adds the window's partial by log-sum-exp.  A
 * context that the window covers (T <= n_s + n_r) reads no packed rows. */
int blockgtq_decode_attn_protected(const bgtq_config* cfg, const void* d_layout, int32_t layer, const void* d_q,
                                   const int32_t* d_ctx_len, int32_t max_ctx, const bgtq_cache* cache,
                                   const void* d_window, int32_t n_sink, int32_t n_recent, float* d_out,
                                   void* d_workspace, size_t ws_bytes, int32_t n_splits, void* stream);

/* ---- (f2) decode step from pre-RoPE inputs --------------------------------
 * One decode step of every layer with RoPE applied on the device (Sec. 2.1:
 * block i = dims (i, i + 64) of a vector at position t is rotated by the angle
 * t * theta_i, theta_i = rope_base^(-2i/d_h); Sec. 2.3, the absolute rotation
 * R_t).  The angle is formed and reduced in fp64.  Three launches on `stream`,
 * no allocation, no memset, so the step can be captured in a HIP graph and
 * replayed with new inputs written into the same buffers:
 *   1. RoPE of the query and key rows at position d_pos[b], into fp32
 *      workspace rows (the value row is copied to fp32 beside them), and
 *      ctx[b] = d_pos[b] + 1;
 *   2. blockgtq_quantize_append of the rotated key and the value at row
 *      d_pos[b] of every layer;
 *   3. blockgtq_decode_attn of every layer over rows [0, d_pos[b] + 1).
 * d_q_pre: pre-RoPE queries [n_layers][batch][n_kv_heads*group][128],
 * d_k_pre, d_v: [n_layers][batch][1][n_kv_heads][128], all in in_dtype.
 * d_pos: device int32 [batch], the new row's position; the caller keeps
 *      d_pos[b] < capacity (rows past it are not written) and max_ctx >=
 *      every d_pos[b] + 1 (it sizes the splits); a sequence whose d_pos[b] + 1
 *      exceeds max_ctx, or whose d_pos[b] is negative, gets NaN outputs, as in
 *      blockgtq_decode_attn.
 * rope_base: theta base, finite and > 1 (EINVAL otherwise).
 * d_out: float [n_layers][batch][n_kv_heads*group][128].
 * d_workspace: blockgtq_rope_step_workspace_bytes; its first part is a
 *      blockgtq_decode_attn workspace (zero-filled once before first use). */
int blockgtq_rope_step_workspace_bytes(const bgtq_config* cfg, int32_t max_ctx, int32_t n_splits,
                                       size_t* bytes_out);
int blockgtq_rope_decode_step(const bgtq_config* cfg, const void* d_layout, double rope_base, const void* d_q_pre,
                              const void* d_k_pre, const void* d_v, const int32_t* d_pos, int32_t max_ctx,
                              const bgtq_cache* cache, float* d_out, void* d_workspace, size_t ws_bytes,
                              int32_t n_splits, void* stream);

/* ---- Decode attention that allocates nothing ---------------------------------
 * For callers that cannot allocate device memory or pass a workspace: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same computation, arguments and results as
 * blockgtq_decode_attn (bit-identical for the same n_splits), except that
 * the split counters and partials live in a static device array of
 * BGTQ_NOALLOC_SCRATCH_BYTES bytes per GPU (held until the process ends; its
 * address is looked up on the first call on each device).  Two launches on
 * `stream`: a fill kernel that zeroes the counters, then the decode.  A
 * call whose workspace (blockgtq_workspace_bytes for the same arguments)
 * exceeds the array fails with BGTQ_EWORKSPACE before anything is enqueued.
 * No hipMalloc / hipFree or allocating library call is made.  Calls that
 * overlap in time on one GPU share the array and race: the caller serialises
 * them (one stream, or events). */
#define BGTQ_NOALLOC_SCRATCH_BYTES (8u << 20)
int blockgtq_decode_attn_noalloc(const bgtq_config* cfg, const void* d_layout, int32_t layer, const void* d_q,
                                 const int32_t* d_ctx_len, int32_t max_ctx, const bgtq_cache* cache, float* d_out,
                                 int32_t n_splits, void* stream);

/* ---- Measurement helper (not a step of the method) ------------------------
 * Streaming read of d_src[0 .. bytes): the read-bandwidth ceiling that the
 * decode's roofline fraction is quoted against, next to the nominal 8 TB/s
 * of HBM3E.  Async on `stream`.  bytes: a positive multiple of 16, d_src
 * 16-byte aligned (EINVAL otherwise).  d_sink: device uint32[1], written only
 * when the folded words equal a fixed constant (the loads stay live). */
int blockgtq_read_probe(const void* d_src, size_t bytes, uint32_t* d_sink, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* BLOCKGTQ_H */
