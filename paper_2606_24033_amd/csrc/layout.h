// Device-resident layout blob shared by the host setup code and the kernels.
//
// The blob holds every constant of the packed cache: the fp16 codebooks and
// decision thresholds of the scalar quantizer (TQ-MSE, Sec. 2.2), the shared
// rotations, and per (layer, KV head) the same-rate grouping of the key row
// (end of Sec. 3.2) flattened into per-position tables.
#pragma once
#include <stdint.h>

namespace bgtq {

constexpr int kHeadDim = 128;        // d_h
constexpr int kBlocks = 64;          // L = d_h / 2 RoPE blocks
constexpr int kTile = 32;            // tokens per value tile
constexpr int kKeyTile = 64;         // tokens per decode tile; the capacity is a multiple of it
constexpr int kMaxGroups = 8;        // same-rate groups (b = 1..8)
constexpr int kMaxKWords = 32;       // 128 positions x 8 bits / 32
constexpr int kMaxSteps = 48;        // 4-coordinate decode steps of a key row (<= 32 + 8)
constexpr int kCodebookEntries = 510;   // sum_b 2^b, b = 1..8
constexpr int kThresholdEntries = 502;  // sum_b (2^b - 1)
constexpr int kRotKFloats = 357760;     // sum over d = 2..128 (even) of d*d
constexpr uint32_t kMagic = 0x51544742u;  // "BGTQ"

__host__ __device__ constexpr int cb_index(int b) { return (1 << b) - 2; }
__host__ __device__ constexpr int thr_index(int b) { return (1 << b) - 1 - b; }
// float offset of the d x d K rotation inside the K rotation block
__host__ __device__ constexpr int rotk_index(int d) {
  // sum_{e=2,4,..,d-2} e^2 = 4 * sum_{m=1}^{d/2-1} m^2
  return 4 * ((d / 2 - 1) * (d / 2) * (d - 1) / 6);
}

// Per (layer, KV head) description of one key row (stream order).
//
// Decode steps: the attention kernel consumes a key row 4 coordinates at a
// time, never mixing two groups in one step (a group with d_g = 2 mod 4 ends
// with a 2-coordinate step).  step[s] packs:
//   bits  0..9  stream bit offset of the step's first code
//   bits 10..13 code width b
//   bits 14..16 group ordinal
//   bit  17     last step of its group
//   bits 19..25 stream position of the step's first coordinate
//   bits 26..28 valid coordinates (2 or 4)
struct RowMeta {
  uint8_t dim[kHeadDim];       // stream position -> source dim of the key
  uint8_t width[kHeadDim];     // code width of the position (bits)
  uint16_t bitoff[kHeadDim];   // first bit of the position's code in the row
  uint8_t grp[kHeadDim];       // group ordinal of the position
  int32_t n_groups;
  int32_t g_bits[kMaxGroups];  // width of group g
  int32_t g_dim[kMaxGroups];   // d_g = 2 |G_b|
  int32_t g_pos[kMaxGroups];   // first stream position of group g
  int32_t word_first[kMaxKWords];  // first position whose code touches word w
  uint32_t step[kMaxSteps];
  int32_t n_steps;
  int32_t word_step[kMaxKWords + 1];  // steps starting in word w: [word_step[w], word_step[w+1])
  // packed decode metadata by width b (entry b - 1; 0 = width absent): bit 31
  // present, bits 0..9 first stream bit, 10..15 steps, 16..19 first query
  // slot (16 steps per slot, slots numbered group after group), 20..22 the
  // group ordinal, 23 hi part of the query only (a width <= 2 group in a row
  // that also holds codes of 4 bits or more)
  uint32_t gm[8];
  int32_t pad[13];
};
static_assert(sizeof(RowMeta) == 1280, "RowMeta size");

struct Header {
  uint32_t magic;
  int32_t n_rows;        // n_layers * n_kv_heads
  int32_t n_kv_heads;
  int32_t k_words;
  int32_t v_bits;
  int32_t pad0[3];
  uint64_t off_c16;      // uint16 [510]   fp16 centroids, b-th table at cb_index(b)
  uint64_t off_thr;      // float  [502]   thresholds, b-th table at thr_index(b)
  uint64_t off_rotv;     // float  [128][128] Pi_V row-major
  uint64_t off_rotvt;    // float  [128][128] Pi_V transposed
  uint64_t off_rotkt;    // float  [kRotKFloats] each Pi_d transposed, at rotk_index(d)
  uint64_t off_rows;     // RowMeta [n_rows]
  uint64_t total_bytes;
  uint64_t off_order;    // int32 [2][n_rows]  row dispatch orders (see layout_order_offset)
  uint64_t off_rowrot;   // float [n_rows][kRowRotFloats] per-row group rotations
  uint64_t pad1[3];
};
static_assert(sizeof(Header) == 128, "Header size");

// Byte offsets of the blob's sections (fixed; only the RowMeta count varies).
__host__ __device__ constexpr uint64_t align256(uint64_t x) { return (x + 255) & ~uint64_t(255); }
constexpr uint64_t kOffC16 = align256(sizeof(Header));
constexpr uint64_t kOffThr = align256(kOffC16 + 2 * kCodebookEntries);
constexpr uint64_t kOffRotV = align256(kOffThr + 4 * kThresholdEntries);
constexpr uint64_t kOffRotVT = align256(kOffRotV + 4 * kHeadDim * kHeadDim);
constexpr uint64_t kOffRotKT = align256(kOffRotVT + 4 * kHeadDim * kHeadDim);
constexpr uint64_t kOffRows = align256(kOffRotKT + 4ull * kRotKFloats);
// After the row metadata:
//  * two int32 [n_rows] dispatch orders of the rows, most expensive decode
//    first (an estimate from the group widths): over all rows (entries are
//    row indices), then per layer (entries are KV-head indices);
//  * per row, its groups' rotations Pi_dg (transposed, as at rotk_index) one
//    after the other, at a fixed stride of kRowRotFloats floats, so that a
//    kernel can address them from the row index alone.
constexpr int kRowRotFloats = kHeadDim * kHeadDim;
__host__ __device__ constexpr uint64_t layout_order_offset(int n_rows) {
  return align256(kOffRows + sizeof(RowMeta) * static_cast<uint64_t>(n_rows));
}
__host__ __device__ constexpr uint64_t layout_rowrot_offset(int n_rows) {
  return align256(layout_order_offset(n_rows) + 8ull * static_cast<uint64_t>(n_rows));
}
// Then the operands of the prefill quantize kernels (quantize.hip), in the
// order the fp32 16x16x4 MFMAs read them: matrix M (128 x 128) is stored as
// [t][s4][lane][e] = M[16 t + lane % 16][32 (lane / 16) + 4 s4 + e], so that
// lane l's float4 at ((t * 8 + s4) * 64 + l) is its operand for the four
// k-steps 4 s4 .. 4 s4 + 3 of output tile t (k-step s of lane l pairs with
// input dim 32 (l / 16) + s):
//  * once: Pi_V;
//  * per row: its key rotation on the input's natural dims, W[p][d] =
//    Pi_g[j][k] for stream position p = g_pos + j and dim d = dim[g_pos + k]
//    of the same group g, zero elsewhere (the gather into stream order is
//    folded into the matrix).
constexpr int kMfmaMatFloats = kHeadDim * kHeadDim;
__host__ __device__ constexpr uint64_t layout_rotv_mfma_offset(int n_rows) {
  return align256(layout_rowrot_offset(n_rows) + 4ull * kRowRotFloats * static_cast<uint64_t>(n_rows));
}
__host__ __device__ constexpr uint64_t layout_kdense_offset(int n_rows) {
  return layout_rotv_mfma_offset(n_rows) + 4ull * kMfmaMatFloats;
}
__host__ __device__ constexpr uint64_t layout_total_bytes(int n_rows) {
  return layout_kdense_offset(n_rows) + 4ull * kMfmaMatFloats * static_cast<uint64_t>(n_rows);
}
// index of M[r][c] in the MFMA operand order above
__host__ __device__ constexpr int mfma_mat_index(int r, int c) {
  return (((r >> 4) * 8 + ((c & 31) >> 2)) * 64 + (c >> 5) * 16 + (r & 15)) * 4 + (c & 3);
}

}  // namespace bgtq
