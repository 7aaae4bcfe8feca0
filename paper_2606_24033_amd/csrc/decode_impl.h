// Packed-cache decode attention for gfx950 in one kernel (Sec. 4: Q-side
// rotation, then fused unpack -> codebook -> norm rescale -> QK and PV
// products -> online softmax over a split of the key axis, then the exact
// log-sum-exp merge of the splits and the inverse V rotation).
//
// Work mapping.  One workgroup (one per CU: the lookup tables fill its LDS;
// 16 waves for up to 4 query heads per KV head, 12 for 5-8) = one (split,
// KV head, sequence[, layer]).  A wave owns 64-token tiles (two value
// tiles).  Both products run
// on 4x4x4 f16 MFMA instructions (16 independent 4x4 blocks) whose A operand
// is broadcast from one block (CBSZ = 4, ABID = the block), so the operand
// shared by all 64 lanes is held once per 16 steps instead of once per step:
//  * QK  D_b = A x B_b.  A = 4 rotated-query heads x 4 coordinates of one
//    decode step, taken from block ABID = step % 16 of a register image in
//    which lane 4b+i holds step b of a 16-step slot for head i.
//    B_b column j = the 4 dequantized coordinates of token 4b+j: lane l
//    decodes the key row of token l, 4 stream positions per step.  All lanes
//    decode the same positions in a step, so they share one code width and a
//    step never mixes two groups.  D lands as lane = token, register = head.
//    A group's partial dot products are scaled by its fp16 radius in fp32.
//  * PV  A = the softmax weights of 4 heads x 4 tokens (block ABID = 4-token
//    step), B_b column j = 4 dequantized value codes of dim 64h + 4b + j,
//    decoded straight from the value tile (the codes of one coordinate are
//    contiguous there).  D lands as lane = dim, register = head.
// Between the two, a 4x4 transpose inside each lane quad turns (token, head)
// into (head, 4 tokens), the layout of the PV A operand and of the softmax.
//
// Same-rate groups have distinct widths, so the QK loop is unrolled over the
// width b = 1..8 (absent widths skipped by a uniform branch): the width, the
// lookup table and the register that holds the group radius are compile-time
// constants.  A group's steps are processed in sub-chunks of 8 (b <= 4) or 4
// steps whose bits are first realigned to bit 0 of a small word array; inside
// a sub-chunk all table lookups are issued before the first MFMA that needs
// them (two passes entered at the step count, so no step is padded).
//
// Dequantization goes through lookup tables in LDS, replicated per lane so
// random indices rarely collide on a bank: 4 codes per lookup for b <= 2 (a
// 64-bit entry of four fp16 centroids), 2 codes for b = 3, 4, 1 code above.
// The rotated query is split into fp16 hi and lo parts (both multiplied,
// accumulated in fp32): fp16 alone leaves ~2^-12 relative error per term.
// 1- and 2-bit groups of rows that also hold codes of 4 bits or more take
// the hi part only.
#pragma once
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <type_traits>
#include <utility>

#include "kernels.h"
#include "layout.h"

namespace bgtq {
namespace split_detail {

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kWaves = 16;  // the 16-wave workgroup (merge-area sizes, the one-set decode)
constexpr int kThreads = kWaves * 64;
// Waves of a packed-decode workgroup: 16 (4 per SIMD) with one query set;
// 12 with two (3 per SIMD, up to 168 VGPRs for the doubled accumulators:
// -10 to -13 % decode time against 16 waves that spill, measured at 128K and
// 512K rows).
template <int NSET>
constexpr int split_waves() { return NSET == 1 ? 16 : 12; }
constexpr int kMaxSlots = 10;  // 16-step query slots of one key row: sum_g ceil(steps_g / 16)
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLog2e = 1.4426950408889634f;
// 2^x (the hardware exponential; arguments here are <= 0)
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }
// A quiet NaN the compiler cannot see (these files are built assuming no
// NaNs): the output scale of a sequence whose context length is out of range.
__device__ __forceinline__ float opaque_nan() {
  uint32_t b = 0x7FC00000u;
  asm volatile("" : "+v"(b));
  return __uint_as_float(b);
}
// fp16(p0 lo(w)) | fp16(p1 hi(w)) << 16, w = two fp16: one mixed-precision
// fused product into each half (single rounding to fp16)
__device__ __forceinline__ uint32_t mix_pair(float p0, float p1, uint32_t w) {
  uint32_t r;
  asm("v_fma_mixlo_f16 %0, %1, %2, 0 op_sel_hi:[0,1,0]" : "=v"(r) : "v"(p0), "v"(w));
  asm("v_fma_mixhi_f16 %0, %1, %2, 0 op_sel:[0,1,0] op_sel_hi:[0,1,0]" : "+v"(r) : "v"(p1), "v"(w));
  return r;
}

// LDS map (bytes).  The b = 2 table has 32 replicas at a 256-byte entry
// stride: the lanes of a half-wave read 32 distinct banks, and the address is
// one byte permute of (code byte, replica offset).  Other entry strides: 128 B
// for the 16- and 32-replica tables, 32 B for the 8-replica b = 4 table, 2 B
// for the plain b >= 6 tables.  Every table starts at a multiple of its own
// size, so an address is (entry << stride) | (table base + replica offset):
// one shift and one and-or per lookup.
constexpr int kLut2 = 0;                        // b=2: 256 entries (4 codes) x 32 replicas x 8 B
constexpr int kLut1B = kLut2 + 256 * 256;       // b=1 keys: 256 entries (8 codes) x 8 replicas x 16 B
constexpr int kLut3 = kLut1B + 256 * 8 * 16;    // b=3: 64 (2 codes) x 32 x 4
constexpr int kLut4 = kLut3 + 64 * 32 * 4;      // b=4: 256 (2 codes) x 8 x 4
constexpr int kLut5 = kLut4 + 256 * 8 * 4;      // b=5: 32 (1 code, low half) x 32 x 4
constexpr int kLut1 = kLut5 + 32 * 32 * 4;      // b=1 values: 16 entries (4 codes) x 16 replicas x 8 B
constexpr int kLutF = kLut1 + 16 * 16 * 8;      // b=8,7,6: plain fp16 tables at +0, +512, +768
constexpr int kQimg = kLutF + 1024;             // [slot][set][hi,lo][lane] x 8 B
static_assert(kLut1B % 32768 == 0 && kLut3 % 8192 == 0 && kLut4 % 8192 == 0 && kLut5 % 4096 == 0 &&
                  kLut1 % 2048 == 0 && kLutF % 1024 == 0,
              "table alignment");
template <int B>
constexpr int lutf_base() { return kLutF + (B == 8 ? 0 : (B == 7 ? 512 : 768)); }
constexpr int kQimgBytes = kMaxSlots * 2 * 2 * 64 * 8;
constexpr int kGmeta = kQimg + kQimgBytes;      // flag word of the split merge
constexpr int kCbStage = kGmeta + 64;           // fp16 codebooks, staged for the table build
constexpr int kLdsBytes = kCbStage + 2 * 512;
static_assert(2 * kCodebookEntries <= 2 * 512, "codebook staging");
static_assert(kLdsBytes <= 160 * 1024, "one workgroup per CU");

// Packed group metadata, indexed by width: bit 31 present, bits 0..9 first
// stream bit, 10..15 steps, 16..19 first query slot, 20..22 radius plane.
__device__ __forceinline__ int gm_off(uint32_t gm) { return gm & 1023; }
__device__ __forceinline__ int gm_steps(uint32_t gm) { return (gm >> 10) & 63; }
__device__ __forceinline__ int gm_slot(uint32_t gm) { return (gm >> 16) & 15; }
__device__ __forceinline__ int gm_plane(uint32_t gm) { return (gm >> 20) & 7; }

__device__ __forceinline__ uint32_t lds32(const uint8_t* s, uint32_t off) {
  return *reinterpret_cast<const uint32_t*>(s + off);
}
__device__ __forceinline__ uint2 lds64(const uint8_t* s, uint32_t off) {
  return *reinterpret_cast<const uint2*>(s + off);
}
__device__ __forceinline__ uint32_t lds16(const uint8_t* s, uint32_t off) {
  return *reinterpret_cast<const uint16_t*>(s + off);
}
__device__ __forceinline__ half4_t as_half4(uint32_t lo, uint32_t hi) {
  return __builtin_bit_cast(half4_t, make_uint2(lo, hi));
}
__device__ __forceinline__ float ld_q(const void* q, size_t i, int dtype) {  // BGTQ_BF16 = 1
  if (dtype == 1) return __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(q)[i]) << 16);
  return reinterpret_cast<const float*>(q)[i];
}
__device__ __forceinline__ float h2f(uint32_t bits16) {
  return __half2float(__ushort_as_half(static_cast<unsigned short>(bits16)));
}

// quad_perm DPP move of a 32-bit value (ctrl = p0 | p1<<2 | p2<<4 | p3<<6)
template <int CTRL>
__device__ __forceinline__ float qperm(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// 4x4 transpose inside every lane quad: on entry lane p of a quad holds
// x[r] = M[r][p]; on exit it holds x[t] = M[p][t].  Two exchange stages
// (partner lanes p ^ 1, then p ^ 2); each output element is one select whose
// other operand is read from the partner lane by DPP (v_cndmask_b32 takes the
// DPP operand as src0, chosen where the lane mask in vcc is clear).  The
// s_nop 1 lines give the two wait states a DPP read needs after a VALU
// write of its operand.
__device__ __forceinline__ void quad_transpose(float4_t& x, int) {
  float y0, y1, y2, y3, z0, z1, z2, z3;
  asm volatile(
      // stage 1: even lanes take x1, x3 from the odd partner's x0, x2; odd
      // lanes take x0, x2 from the even partner's x1, x3
      "s_mov_b32 vcc_lo, 0x55555555\n\t"
      "s_mov_b32 vcc_hi, 0x55555555\n\t"
      "s_nop 1\n\t"
      "v_cndmask_b32_dpp %0, %5, %4, vcc quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_cndmask_b32_dpp %2, %7, %6, vcc quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "s_not_b64 vcc, vcc\n\t"
      "v_cndmask_b32_dpp %1, %4, %5, vcc quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_cndmask_b32_dpp %3, %6, %7, vcc quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf"
      : "=&v"(y0), "=&v"(y1), "=&v"(y2), "=&v"(y3)
      : "v"(x[0]), "v"(x[1]), "v"(x[2]), "v"(x[3])
      : "vcc");
  asm volatile(
      // stage 2: lanes 0, 1 of a quad take x2, x3 from partner p + 2's x0,
      // x1; lanes 2, 3 take x0, x1 from partner p - 2's x2, x3
      "s_mov_b32 vcc_lo, 0x33333333\n\t"
      "s_mov_b32 vcc_hi, 0x33333333\n\t"
      "s_nop 1\n\t"
      "v_cndmask_b32_dpp %0, %6, %4, vcc quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
      "v_cndmask_b32_dpp %1, %7, %5, vcc quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
      "s_not_b64 vcc, vcc\n\t"
      "v_cndmask_b32_dpp %2, %4, %6, vcc quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
      "v_cndmask_b32_dpp %3, %5, %7, vcc quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf"
      : "=&v"(z0), "=&v"(z1), "=&v"(z2), "=&v"(z3)
      : "v"(y0), "v"(y1), "v"(y2), "v"(y3)
      : "vcc");
  x = float4_t{z0, z1, z2, z3};
}

// Rotate right by N lanes inside every 16-lane row (DPP row_ror).
template <int N>
__device__ __forceinline__ float row_ror(float v) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x120 + N, 0xF, 0xF, false));
}
// Lane swaps of gfx950: r0, r1 = the values of rows 2k and 2k+1 (16-lane
// rows) at this lane's row position, resp. of lanes l % 32 and l % 32 + 32.
// Written as inline asm with both registers as outputs: the compiler's
// builtin for these instructions returns the first register twice.  The
// s_nop pairs cover the VALU-to-permlane operand hazard on either side.
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
// Max / sum over the 16 lanes with equal (lane & 3); every lane gets the
// same result (the cross-row steps combine rows in a fixed order).
__device__ __forceinline__ float xmax16(float v) {
  float a, b;
  v = fmaxf(v, row_ror<4>(v));
  v = fmaxf(v, row_ror<8>(v));
  swap16(v, a, b);
  swap32(fmaxf(a, b), a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float xsum16(float v) {
  float a, b;
  v += row_ror<4>(v);
  v += row_ror<8>(v);
  swap16(v, a, b);
  swap32(a + b, a, b);
  return a + b;
}

// Bits [POS, POS + LEN) of the little-endian word array w, placed at bit SH
// (other bits zero): one shift (or funnel shift) and one mask.
template <int POS, int LEN, int SH, int N>
__device__ __forceinline__ uint32_t field_at(const uint32_t (&w)[N]) {
  constexpr int wi = POS / 32, sh = POS % 32;
  static_assert(wi < N && SH + LEN <= 32, "field");
  uint32_t v;
  if constexpr (sh + LEN > 32) {
    static_assert(wi + 1 < N && sh >= SH, "field word");
    v = __builtin_amdgcn_alignbit(w[wi + 1], w[wi], sh - SH);
  } else if constexpr (sh >= SH) {
    v = w[wi] >> (sh - SH);
  } else {
    v = w[wi] << (SH - sh);
  }
  return v & (((1u << LEN) - 1u) << SH);
}

// Per-lane table base + replica offset of each lookup table.
struct LaneRep {
  uint32_t r1;   // kLut1 + (lane & 15) * 8
  uint32_t r3;   // kLut3 + (lane & 31) * 4
  uint32_t r4;   // kLut4 + (lane & 7) * 4
  uint32_t r5;   // kLut5 + (lane & 31) * 4
  uint32_t r2;   // kLut2 + (lane & 31) * 8
  uint32_t r1b;  // kLut1B + (lane & 7) * 16, or kLut1B (the 12-bit table, kernels of 3-bit values)
  uint32_t qimg; // kQimg + lane * 8: this lane's entry in slot 0 of the query image
};

// Byte K of w (a compile-time byte) as the entry index of the b = 2 table:
// one permute builds entry * 256 + replica.
template <int K>
__device__ __forceinline__ uint32_t lut2_addr(uint32_t w, uint32_t r2) {
  return __builtin_amdgcn_perm(w, r2, 0x0C0C0000u | ((4u + K) << 8));
}

// Four consecutive B-bit codes starting at bit POS of w -> four fp16
// centroids (an MFMA operand).
template <int B, int POS, bool T12, int N>
__device__ __forceinline__ half4_t decode4(const uint8_t* smem, const uint32_t (&w)[N], const LaneRep& r) {
  if constexpr (B == 2 && POS % 8 == 0) {
    const uint2 u = lds64(smem, lut2_addr<(POS % 32) / 8>(w[POS / 32], r.r2));
    return as_half4(u.x, u.y);
  } else if constexpr (B == 2) {
    const uint2 u = lds64(smem, field_at<POS, 8, 8>(w) | r.r2);
    return as_half4(u.x, u.y);
  } else if constexpr (B == 1) {
    const uint2 u = lds64(smem, field_at<POS, 4, 7>(w) | r.r1);
    return as_half4(u.x, u.y);
  } else if constexpr (B == 3 && T12) {
    // the 12-bit table: four codes, one lookup (r.r1b holds its base)
    const uint2 u = lds64(smem, field_at<POS, 12, 3>(w) | r.r1b);
    return as_half4(u.x, u.y);
  } else if constexpr (B == 3) {
    return as_half4(lds32(smem, field_at<POS, 6, 7>(w) | r.r3), lds32(smem, field_at<POS + 6, 6, 7>(w) | r.r3));
  } else if constexpr (B == 4) {
    return as_half4(lds32(smem, field_at<POS, 8, 5>(w) | r.r4), lds32(smem, field_at<POS + 8, 8, 5>(w) | r.r4));
  } else {
    constexpr int LS = B == 5 ? 7 : 1;
    const uint32_t rb = B == 5 ? r.r5 : static_cast<uint32_t>(lutf_base<B>());
    const uint32_t c0 = lds16(smem, field_at<POS, B, LS>(w) | rb);
    const uint32_t c1 = lds16(smem, field_at<POS + B, B, LS>(w) | rb);
    const uint32_t c2 = lds16(smem, field_at<POS + 2 * B, B, LS>(w) | rb);
    const uint32_t c3 = lds16(smem, field_at<POS + 3 * B, B, LS>(w) | rb);
    return as_half4(c0 | (c1 << 16), c2 | (c3 << 16));
  }
}

// ---------------------------------------------------------------- QK
template <int B>
constexpr int qk_ch() { return B <= 4 ? 8 : 4; }           // steps per sub-chunk
constexpr int kRowPad = 4;  // zero words after a key row: a sub-chunk reads words w0 .. w0 + 4
template <int B>
constexpr int qk_nw() { return (qk_ch<B>() * 4 * B + 31) / 32; }  // words per sub-chunk

// One MFMA pair (hi and lo query parts) of query block K; LO = false leaves
// out the lo part (1-bit groups: their terms are the smallest, see below).
template <int NSET, int K, bool LO = true, bool Z = false>
__device__ __forceinline__ void qk_mac(const half4_t& kv, const half4_t (&qh)[NSET], const half4_t (&ql)[NSET],
                                       float4_t (&acc)[NSET]) {
#pragma unroll
  for (int s = 0; s < NSET; ++s) {
    if constexpr (Z)  // the group's first product starts its accumulator
      acc[s] = __builtin_amdgcn_mfma_f32_4x4x4f16(qh[s], kv, float4_t{0.f, 0.f, 0.f, 0.f}, 4, K, 0);
    else
      acc[s] = __builtin_amdgcn_mfma_f32_4x4x4f16(qh[s], kv, acc[s], 4, K, 0);
    if constexpr (LO) acc[s] = __builtin_amdgcn_mfma_f32_4x4x4f16(ql[s], kv, acc[s], 4, K, 0);
  }
}

// Window W (steps 4W..4W+3) of a sub-chunk whose first step uses query
// block K0; steps >= mm do not exist.  For b <= 4 the four lookups are
// issued unconditionally (a step past the group end decodes other bits of
// the row or its zero padding: a valid table index, whose MFMA is skipped),
// so the decoded operands need no merge copies; wider codes take four
// lookups a step and are decoded only when the step exists.
template <int B, int NSET, bool T12, int K0, int W, int N, bool Z, bool HI>
__device__ __forceinline__ void qk_window(const uint8_t* smem, const uint32_t (&aw)[N], int mm, const LaneRep& rep,
                                          const half4_t (&qh)[NSET], const half4_t (&ql)[NSET],
                                          float4_t (&acc)[NSET]) {
  constexpr int k = 4 * W;
  if constexpr (B == 1 && !T12) {
    // one 16-byte lookup per code byte: the operands of two steps.  HI: the
    // hi query part only (see qk_group)
    constexpr int by = k / 2;  // byte of step k
    const uint4 u01 = *reinterpret_cast<const uint4*>(smem + (field_at<8 * by, 8, 7>(aw) | rep.r1b));
    const uint4 u23 = *reinterpret_cast<const uint4*>(smem + (field_at<8 * (by + 1), 8, 7>(aw) | rep.r1b));
    half4_t kv0 = as_half4(u01.x, u01.y), kv1 = as_half4(u01.z, u01.w);
    half4_t kv2 = as_half4(u23.x, u23.y), kv3 = as_half4(u23.z, u23.w);
    asm volatile("" : "+v"(kv0), "+v"(kv1), "+v"(kv2), "+v"(kv3));
    qk_mac<NSET, K0 + k, !HI, Z>(kv0, qh, ql, acc);
    if (mm > k + 1) {
      qk_mac<NSET, K0 + k + 1, !HI>(kv1, qh, ql, acc);
      if (mm > k + 2) {
        qk_mac<NSET, K0 + k + 2, !HI>(kv2, qh, ql, acc);
        if (mm > k + 3) qk_mac<NSET, K0 + k + 3, !HI>(kv3, qh, ql, acc);
      }
    }
  } else if constexpr (B <= 4) {
    half4_t kv0 = decode4<B, 4 * B * (k + 0), T12>(smem, aw, rep);
    half4_t kv1 = decode4<B, 4 * B * (k + 1), T12>(smem, aw, rep);
    half4_t kv2 = decode4<B, 4 * B * (k + 2), T12>(smem, aw, rep);
    half4_t kv3 = decode4<B, 4 * B * (k + 3), T12>(smem, aw, rep);
    // keep the four lookups ahead of the guarded products (one LDS round
    // trip per window): without this the compiler sinks each lookup into
    // the branch that uses it and serialises them
    asm volatile("" : "+v"(kv0), "+v"(kv1), "+v"(kv2), "+v"(kv3));
    constexpr bool LO = !HI;
    qk_mac<NSET, K0 + k, LO, Z>(kv0, qh, ql, acc);
    if (mm > k + 1) {
      qk_mac<NSET, K0 + k + 1, LO>(kv1, qh, ql, acc);
      if (mm > k + 2) {
        qk_mac<NSET, K0 + k + 2, LO>(kv2, qh, ql, acc);
        if (mm > k + 3) qk_mac<NSET, K0 + k + 3, LO>(kv3, qh, ql, acc);
      }
    }
  } else {
    qk_mac<NSET, K0 + k, true, Z>(decode4<B, 4 * B * k, T12>(smem, aw, rep), qh, ql, acc);
    if (mm > k + 1) {
      qk_mac<NSET, K0 + k + 1>(decode4<B, 4 * B * (k + 1), T12>(smem, aw, rep), qh, ql, acc);
      if (mm > k + 2) {
        qk_mac<NSET, K0 + k + 2>(decode4<B, 4 * B * (k + 2), T12>(smem, aw, rep), qh, ql, acc);
        if (mm > k + 3) qk_mac<NSET, K0 + k + 3>(decode4<B, 4 * B * (k + 3), T12>(smem, aw, rep), qh, ql, acc);
      }
    }
  }
}

// Sub-chunk SC of a 16-step slot: realign its bits (stream bit ob onwards)
// to bit 0 of aw, then run its min(CH, ms - SC CH) steps.
template <int B, int NSET, bool T12, int KWB, bool Z, bool HI, int SC>
__device__ __forceinline__ void qk_slot_part(const uint8_t* smem, const uint32_t (&rw)[KWB + kRowPad], int ob, int ms,
                                             const LaneRep& rep, const half4_t (&qh)[NSET],
                                             const half4_t (&ql)[NSET], float4_t (&acc)[NSET]) {
  constexpr int CH = qk_ch<B>(), NW = qk_nw<B>();
  // (with Z, sub-chunk 0 always exists: a group has at least one step)
  if ((Z && SC == 0) || SC * CH < ms) {
    const int o = ob + SC * CH * 4 * B;
    const int w0 = o >> 5, sh = o & 31;
    uint32_t aw[NW + 1];
#pragma unroll
    for (int i = 0; i < NW; ++i) aw[i] = __builtin_amdgcn_alignbit(rw[w0 + i + 1], rw[w0 + i], sh);
    aw[NW] = 0;
    const int mm = min(CH, ms - SC * CH);
    qk_window<B, NSET, T12, SC * CH, 0, NW + 1, Z && SC == 0, HI>(smem, aw, mm, rep, qh, ql, acc);
    if constexpr (CH == 8) {
      if (mm > 4) qk_window<B, NSET, T12, SC * CH, 1, NW + 1, false, HI>(smem, aw, mm, rep, qh, ql, acc);
    }
  }
}

template <int B, int NSET, bool T12, int KWB, bool Z, bool HI, int... SC>
__device__ __forceinline__ void qk_slot(std::integer_sequence<int, SC...>, const uint8_t* smem,
                                        const uint32_t (&rw)[KWB + kRowPad], int ob, int ms, const LaneRep& rep,
                                        const half4_t (&qh)[NSET], const half4_t (&ql)[NSET], float4_t (&acc)[NSET]) {
  (qk_slot_part<B, NSET, T12, KWB, Z, HI, SC>(smem, rw, ob, ms, rep, qh, ql, acc), ...);
}

// The group of width B (metadata gm, radius bits nrm16 of the lane's token):
// L += radius * <rotated query, dequantized unit-norm codes>.  HI: the hi
// part of the query only, for groups of width <= 2 in rows that also hold
// codes of 4 bits or more (the layout's flag): their blocks are among the
// row's lowest-energy ones, and leaving out their lo products moves the
// attention output by <= 3.4e-4 (relative) on the Llama-shaped workload.  A
// row whose low widths carry most of the energy (a uniform 1- or 2-bit
// layout) keeps both parts: fp16 queries alone cost ~3e-3 there.
template <int B, int NSET, bool T12, int KWB, bool HI>
__device__ __forceinline__ void qk_group(const uint8_t* smem, const uint32_t (&rw)[KWB + kRowPad], uint32_t gm,
                                         uint32_t nrm16, const LaneRep& rep, int lane, float4_t (&L)[NSET]) {
  const int o = gm_off(gm), nst = gm_steps(gm), slot0 = gm_slot(gm);
  float4_t acc[NSET];
  // slot 0 is peeled: its first product writes the accumulator
  const auto slot = [&](auto first, int c) {
    half4_t qh[NSET], ql[NSET];
#pragma unroll
    for (int s = 0; s < NSET; ++s) {
      const uint32_t base = rep.qimg + ((slot0 + c) * 2 + s) * 2 * 64 * 8;  // slot offset: one add
      const uint2 uh = lds64(smem, base), ul = lds64(smem, base + 64 * 8);
      qh[s] = as_half4(uh.x, uh.y);
      ql[s] = as_half4(ul.x, ul.y);
    }
    qk_slot<B, NSET, T12, KWB, decltype(first)::value, HI>(std::make_integer_sequence<int, 16 / qk_ch<B>()>{}, smem, rw,
                                                      o + 64 * B * c, min(16, nst - 16 * c), rep, qh, ql, acc);
  };
  slot(std::true_type{}, 0);
  for (int c = 1; c * 16 < nst; ++c) slot(std::false_type{}, c);
  const float nrm = h2f(nrm16);
#pragma unroll
  for (int s = 0; s < NSET; ++s)
#pragma unroll
    for (int r = 0; r < 4; ++r) L[s][r] = fmaf(nrm, acc[s][r], L[s][r]);
}

// ---------------------------------------------------------------- PV
template <int BV>
constexpr int pv_words() { return BV; }

template <int BV, int NSET, bool T12, int S>
__device__ __forceinline__ void pv_step(const uint8_t* smem, const uint32_t (&vw)[4][pv_words<BV>()],
                                        const LaneRep& rep, const half4_t (&pp)[NSET], float4_t (&O)[NSET][2]) {
  constexpr int tau = S >> 3, sp = S & 7;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const half4_t vv = decode4<BV, 4 * BV * sp, T12>(smem, vw[tau * 2 + h], rep);
#pragma unroll
    for (int s = 0; s < NSET; ++s) O[s][h] = __builtin_amdgcn_mfma_f32_4x4x4f16(pp[s], vv, O[s][h], 4, S, 0);
  }
}

template <int BV, int NSET, bool T12, int... S>
__device__ __forceinline__ void pv_steps(std::integer_sequence<int, S...>, const uint8_t* smem,
                                         const uint32_t (&vw)[4][pv_words<BV>()], const LaneRep& rep,
                                         const half4_t (&pp)[NSET], float4_t (&O)[NSET][2]) {
  (pv_step<BV, NSET, T12, S>(smem, vw, rep, pp, O), ...);
}

// ---------------------------------------------------------------- loads
// Load of a T at a 32-bit byte offset from a wave-uniform base (the global
// load form with a scalar base and a 32-bit vector offset).
template <class T>
__device__ __forceinline__ T ld_at(const void* base, uint32_t byte_off) {
  return *reinterpret_cast<const T*>(static_cast<const char*>(base) + byte_off);
}

// Cache rows of one (layer, sequence, KV head).
struct RowPtrs {
  const uint32_t* k;   // [cap][kw] key rows
  const uint16_t* kn;  // [cap][S] group radii, S = n_g rounded up to even
  const uint32_t* v;   // [cap / 32][128][BV] value tiles
  const uint16_t* vn;  // [cap] value radii
};

// Key data of the 64-token tile at t0 (loaded one tile ahead of its use):
// rw[0..kw) = the key row of token t0 + lane (zero up to KWB), knp[g / 2]
// half g & 1 = that token's radius of group ordinal g.  Every token of a
// tile is below the capacity (a multiple of 64).
template <int KWB>
__device__ __forceinline__ void load_keys(uint32_t (&rw)[KWB], uint32_t (&knp)[4], int nslot, const RowPtrs& R,
                                          int kw, int t0, int lane) {
  const uint32_t* src = R.k + static_cast<size_t>(t0) * kw;
  const uint32_t lo = static_cast<uint32_t>(lane * kw * 4);
  if ((kw & 3) == 0) {
#pragma unroll
    for (int i = 0; i < KWB; i += 4) {
      if (i < kw) {
        const uint4 v = ld_at<uint4>(src, lo + 4 * i);
        rw[i] = v.x;
        rw[i + 1] = v.y;
        rw[i + 2] = v.z;
        rw[i + 3] = v.w;
      } else {
        rw[i] = rw[i + 1] = rw[i + 2] = rw[i + 3] = 0u;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < KWB; ++i) rw[i] = i < kw ? ld_at<uint32_t>(src, lo + 4 * i) : 0u;
  }
  const uint16_t* nb = R.kn + static_cast<size_t>(t0) * nslot;
  const uint32_t lo2 = static_cast<uint32_t>(lane * nslot * 2);
  // one 16-byte window per token (slots past n_g belong to the next token and
  // are never used; the window stays inside the row's capacity * 8 slots)
  const uint4 x = ld_at<uint4>(nb, lo2);
  knp[0] = x.x;
  knp[1] = x.y;
  knp[2] = x.z;
  knp[3] = x.w;
}

// Value data of the tile at t0 (loaded when the tile starts, used after its
// QK products): vn = the value radii of tokens t0 + 4(lane/4) .. +3, vw =
// the value words of dims lane and 64 + lane of both value tiles.
template <int BV>
__device__ __forceinline__ void load_values(uint2& vn, uint32_t (&vw)[4][pv_words<BV>()], const RowPtrs& R, int t0,
                                            int lane) {
  vn = ld_at<uint2>(R.vn + t0, static_cast<uint32_t>(8 * (lane >> 2)));
  const uint32_t* vb = R.v + static_cast<size_t>(t0 / kTile) * kHeadDim * BV;
  const uint32_t lo = static_cast<uint32_t>(lane * BV * 4);
#pragma unroll
  for (int th = 0; th < 4; ++th) {
    const uint32_t* src = vb + ((th >> 1) * kHeadDim + 64 * (th & 1)) * BV;
    if constexpr (BV % 4 == 0) {
#pragma unroll
      for (int w = 0; w < BV; w += 4) {
        const uint4 v4 = ld_at<uint4>(src, lo + 4 * w);
        vw[th][w] = v4.x;
        vw[th][w + 1] = v4.y;
        vw[th][w + 2] = v4.z;
        vw[th][w + 3] = v4.w;
      }
    } else if constexpr (BV % 2 == 0) {
#pragma unroll
      for (int w = 0; w < BV; w += 2) {
        const uint2 v2 = ld_at<uint2>(src, lo + 4 * w);
        vw[th][w] = v2.x;
        vw[th][w + 1] = v2.y;
      }
    } else {
#pragma unroll
      for (int w = 0; w < BV; ++w) vw[th][w] = ld_at<uint32_t>(src, lo + 4 * w);
    }
  }
}

// Radius bits of group ordinal g (wave-uniform) from the packed halves.
__device__ __forceinline__ uint32_t radius_bits(const uint32_t (&knp)[4], int g) {
  // g is wave-uniform: one indexed register move, then the half
  return knp[g >> 1] >> (16 * (g & 1));
}

// Radius bits of the group of width BM1 + 1.  Its ordinal is BM1 when every
// narrower width is present, BM1 - 1 when exactly one is missing (rows whose
// narrowest width is 2): in the model-shaped layouts one of the two holds for
// nearly every group of width <= 5, and the radius is then a fixed half of
// knp.  Other groups take the runtime select (uniform branches).
template <int BM1>
__device__ __forceinline__ uint32_t radius_of(const uint32_t (&knp)[4], uint32_t gm) {
  const int g = gm_plane(gm);
  uint32_t r = knp[BM1 >> 1] >> (16 * (BM1 & 1));
  if (g != BM1) {
    asm volatile("" : "+v"(r));  // keeps these branches, not selects on every tile
    if constexpr (BM1 > 0) {
      if (g == BM1 - 1) return knp[(BM1 - 1) >> 1] >> (16 * ((BM1 - 1) & 1));
    }
    r = radius_bits(knp, g);
  }
  return r;
}

// QK of one tile over every present width.
template <int NSET, bool T12, int KWB, int... BM1>
__device__ __forceinline__ void qk_all(std::integer_sequence<int, BM1...>, const uint8_t* smem,
                                       const uint32_t (&rw)[KWB + kRowPad], const uint32_t (&knp)[4],
                                       const uint32_t (&gmb)[8], const LaneRep& rep, int lane, float4_t (&L)[NSET]) {
  // (the hi-only variant exists for widths 1 and 2; the flag is uniform)
  ((gmb[BM1] >> 31 ? (BM1 < 2 && ((gmb[BM1] >> 23) & 1u)
                          ? qk_group<BM1 + 1, NSET, T12, KWB, BM1 < 2>(smem, rw, gmb[BM1], radius_of<BM1>(knp, gmb[BM1]),
                                                                  rep, lane, L)
                          : qk_group<BM1 + 1, NSET, T12, KWB, false>(smem, rw, gmb[BM1], radius_of<BM1>(knp, gmb[BM1]),
                                                                rep, lane, L))
                   : void()),
   ...);
}

// ---------------------------------------------------------------- epilogue
// Merge of the waves' (max, sum, accumulator) states in LDS, then (n_splits
// > 1) of the splits of the unit in the workgroup that finishes it last
// (exact log-sum-exp; it resets the unit's counter), then out = R^T o with R
// the V rotation (rotv) or none, o scaled by oscale.  The merge area of LDS
// starts at smem; `last` is a flag word outside it.
// Log-sum-exp merge of the protected window's partial (m, l, acc[128], written
// by the window kernel before this launch) into a running (mx, l, a).  The
// window's accumulator is in the original V domain: it is added after the
// output rotation, with the weight returned here (its share of the merged
// sum still to be divided by the final l).
__device__ __forceinline__ float merge_window(const float* __restrict__ w, float& mx, float& l, float& a) {
  const float mw = w[0];
  if (mw == kNegInf) return 0.f;
  const float mc = fmaxf(mx, mw);
  const float r = mx == kNegInf ? 0.f : exp2_hw(mx - mc);
  const float e = exp2_hw(mw - mc);
  l = fmaf(w[1], e, l * r);
  a *= r;
  mx = mc;
  return e;
}

template <int NSET, int WAVES>
__device__ __forceinline__ void finish_unit(uint8_t* smem, int* last, const Dims& d, int G, int lz, int kvh,
                                            int split, int tid, int lane, int wave, float (&m_run)[NSET],
                                            float (&l_run)[NSET], const float4_t (&O)[NSET][2],
                                            int32_t* __restrict__ counters, float* __restrict__ part, int n_splits,
                                            float oscale, const float* __restrict__ rotv, float* __restrict__ out,
                                            const float* __restrict__ wpart) {
  const int hqn = d.n_kv * G;
  const int bq = lane >> 2, jq = lane & 3;
#pragma unroll
  for (int s = 0; s < NSET; ++s) l_run[s] = xsum16(l_run[s]);

  // ---------------- merge the waves of the workgroup
  __syncthreads();
  float* fm = reinterpret_cast<float*>(smem);            // [wave][8] max
  float* fl = fm + WAVES * 8;                           // [wave][8] sum
  float* fo = fl + WAVES * 8;                           // [wave][8][128] accumulators
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
  float* os = fo + WAVES * 8 * kHeadDim;  // [G][128] merged output, rotated V domain
  float* ws_ = os + 8 * kHeadDim;          // [G][128] weight of the window's accumulator
  for (int i = tid; i < G * kHeadDim; i += (WAVES * 64)) {
    const int qh = i >> 7, dd = i & 127;
    float mx = kNegInf;
    for (int w = 0; w < WAVES; ++w) mx = fmaxf(mx, fm[w * 8 + qh]);
    float l = 0.f, a = 0.f;
    if (mx != kNegInf) {
      for (int w = 0; w < WAVES; ++w) {
        const float mw = fm[w * 8 + qh];
        if (mw == kNegInf) continue;
        const float e = exp2_hw(mw - mx);
        l = fmaf(fl[w * 8 + qh], e, l);
        a = fmaf(fo[(w * 8 + qh) * kHeadDim + dd], e, a);
      }
    }
    if (n_splits == 1) {
      float e = 0.f;
      if (wpart != nullptr) e = merge_window(wpart + (static_cast<size_t>(lz) * hqn + kvh * G + qh) * 130, mx, l, a);
      os[i] = (l > 0.f ? a / l : 0.f) * oscale;  // oscale NaN: flagged sequence
      if (wpart != nullptr) ws_[i] = l > 0.f ? e / l : 0.f;
    } else {
      // agent-scope stores: written through to the device coherence point
      // (each XCD has its own L2), completed before the counter increment
      // below
      float* pb = part + ((static_cast<size_t>(lz) * hqn + kvh * G + qh) * n_splits + split) * 130;
      __hip_atomic_store(pb + 2 + dd, a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (dd == 0) {
        __hip_atomic_store(pb, mx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(pb + 1, l, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }

  // ---------------- merge the splits (exact log-sum-exp) in the workgroup
  // that finishes last; it resets the counter for the next call
  if (n_splits > 1) {
    // Publication of the partials to the workgroup that merges (possibly on
    // another XCD, with its own L2).  Every partial is written above and read
    // below only by agent-scope atomic accesses, which gfx950 performs at the
    // device coherence point (stores written through, loads not served from
    // a stale L2 line), so no L2 write-back or invalidate is needed; what is
    // needed is the order:
    //  * every wave waits until its own partial stores have completed
    //    (vmcnt(0); the memory clobber keeps the compiler from sinking the
    //    stores below it), then the barrier: all partials of the workgroup
    //    are at the coherence point before the increment is issued;
    //  * thread 0 increments the unit's counter (agent scope) and learns
    //    whether this workgroup finished the unit last;
    //  * only then, behind a barrier, does the last workgroup issue its
    //    loads of the partials.
    // (The agent-scope release / acquire fences would add an L2 write-back
    // per wave and an L2 invalidate: +37 % decode time, measured.)
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0)
      *last = __hip_atomic_fetch_add(counters + lz * d.n_kv + kvh, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
              n_splits - 1;
    __syncthreads();
    if (*last == 0) return;
    for (int i = tid; i < G * kHeadDim; i += (WAVES * 64)) {
      const int qh = i >> 7, dd = i & 127;
      const float* P = part + (static_cast<size_t>(lz) * hqn + kvh * G + qh) * n_splits * 130;
      const auto ld = [](const float* x) { return __hip_atomic_load(x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); };
      // eight splits per round, their loads in flight together; running
      // maximum with rescaling between rounds
      float mx = kNegInf, l = 0.f, a = 0.f;
      for (int sp0 = 0; sp0 < n_splits; sp0 += 8) {
        float ms[8], ls[8], as[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          ms[u] = kNegInf;
          ls[u] = as[u] = 0.f;
          if (sp0 + u < n_splits) {
            const float* ps = P + (sp0 + u) * 130;
            ms[u] = ld(ps);
            ls[u] = ld(ps + 1);
            as[u] = ld(ps + 2 + dd);
          }
        }
        float mc = mx;
#pragma unroll
        for (int u = 0; u < 8; ++u) mc = fmaxf(mc, ms[u]);
        if (mc == kNegInf) continue;
        const float r = mx == kNegInf ? 0.f : exp2_hw(mx - mc);
        l *= r;
        a *= r;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (ms[u] == kNegInf) continue;
          const float e = exp2_hw(ms[u] - mc);
          l = fmaf(ls[u], e, l);
          a = fmaf(as[u], e, a);
        }
        mx = mc;
      }
      float e = 0.f;
      if (wpart != nullptr) e = merge_window(wpart + (static_cast<size_t>(lz) * hqn + kvh * G + qh) * 130, mx, l, a);
      os[i] = (l > 0.f ? a / l : 0.f) * oscale;  // oscale NaN: flagged sequence
      if (wpart != nullptr) ws_[i] = l > 0.f ? e / l : 0.f;
    }
    if (tid == 0) __hip_atomic_store(counters + lz * d.n_kv + kvh, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  // ---------------- out = Pi_V^T o (back from the rotated V domain), or o
  for (int i = tid; i < G * kHeadDim; i += (WAVES * 64)) {
    const int qh = i >> 7, dd = i & 127;
    float r = os[i];
    if (rotv != nullptr) {
      r = 0.f;
      for (int jj = 0; jj < kHeadDim; ++jj) r = fmaf(rotv[jj * kHeadDim + dd], os[qh * kHeadDim + jj], r);
    }
    if (wpart != nullptr) r = fmaf(ws_[i], wpart[(static_cast<size_t>(lz) * hqn + kvh * G + qh) * 130 + 2 + dd], r);
    out[(static_cast<size_t>(lz) * hqn + kvh * G + qh) * kHeadDim + dd] = r;
  }
}

// ---------------------------------------------------------------- kernel
template <int NSET, int KWB, int BV>
__global__ __launch_bounds__(split_waves<NSET>() * 64)
__attribute__((amdgpu_waves_per_eu(NSET == 1 && KWB <= 16 ? 4 : 3))) void k_split_mfma(
    Dims d, const uint8_t* __restrict__ blob, const void* __restrict__ q, const int32_t* __restrict__ ctx_len,
    CachePtrs c, float* __restrict__ out, int32_t* __restrict__ counters, float* __restrict__ part, int n_splits,
    int split_len, WinArgs win) {
  // this instantiation's workgroup (shadows the 16-wave default)
  constexpr int kWaves = split_waves<NSET>(), kThreads = kWaves * 64;
  // kernels of 3-bit values hold the 3-bit codes' 12-bit table (one lookup
  // per four codes, values and keys) where the others hold the 1-bit keys'
  // byte table
  constexpr bool T12 = BV == 3;
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: tile addresses stay scalar
  const int bq = lane >> 2;
  // One-dimensional grid of (unit, split) items, units in the layout's
  // dispatch order (most expensive rows first, so that the second round of
  // workgroups fills in behind the long first ones); the splits of a unit
  // are adjacent.
  const int item = static_cast<int>(__builtin_amdgcn_workgroup_id_x());
  const int split = item % n_splits, rest = item / n_splits;
  const int seq = rest % d.batch, rank = rest / d.batch;
  const int n_rows = d.n_layers * d.n_kv;
  const int32_t* order = reinterpret_cast<const int32_t*>(blob + layout_order_offset(n_rows));
  int layer, kvh;
  if (d.layer >= 0) {
    layer = d.layer;
    kvh = order[n_rows + d.layer * d.n_kv + rank];
  } else {
    const int row = order[rank];
    layer = row / d.n_kv;
    kvh = row - layer * d.n_kv;
  }
  const int lz = d.layer >= 0 ? seq : layer * d.batch + seq;
  const int G = d.group, hqn = d.n_kv * G;
  const int cap = d.capacity, kw = d.k_words;
  const RowMeta* M = reinterpret_cast<const RowMeta*>(blob + kOffRows) + (layer * d.n_kv + kvh);
  const uint16_t* c16 = reinterpret_cast<const uint16_t*>(blob + kOffC16);
  const int ng = M->n_groups;

  // ---- the Q-side rotation (Sec. 4): qr[h][p] = (Pi_g q_g)_j / sqrt(d_g d_h)
  // at stream position p = g_pos[g] + j.  Staged in LDS before the tables
  // are built: the queries as given (qn), the row's group rotations (rs: the
  // blocks Pi_dg transposed, one after the other, at the row's fixed slot in
  // the layout), the stream-position -> dim table and the codebooks.  Every
  // global read of the set-up is issued in one round (none depends on another
  // read's value), then the queries are gathered into stream order (qg) and
  // rotated (qr).
  static_assert((2 * 8 * kHeadDim + kRowRotFloats + 8 * kHeadDim) * 4 + kHeadDim <= kQimg,
                "set-up staging must stay below the query image");
  float* qg = reinterpret_cast<float*>(smem);      // [G][128] queries in stream order
  float* qr = qg + 8 * kHeadDim;                   // [G][128] rotated
  float* rs = qr + 8 * kHeadDim;                   // the row's rotations, <= 128^2 floats
  float* qn = rs + kRowRotFloats;                  // [G][128] queries as given
  uint32_t* dimw = reinterpret_cast<uint32_t*>(qn + 8 * kHeadDim);  // RowMeta::dim
  uint16_t* cbs = reinterpret_cast<uint16_t*>(smem + kCbStage);
  // per-group rotation blocks: staged offset, size, first stream position
  // (whole arrays read, entries past n_g replaced: no load waits on n_g)
  int roff[kMaxGroups], rdim[kMaxGroups], rpos[kMaxGroups];
  int rtot = 0;
#pragma unroll
  for (int g = 0; g < kMaxGroups; ++g) {
    const int a = M->g_dim[g], b = M->g_pos[g];
    rdim[g] = g < ng ? a : 0;
    rpos[g] = g < ng ? b : kHeadDim;
    roff[g] = rtot;
    rtot += rdim[g] * rdim[g];
  }
  {
    constexpr int kRotFirst = kRowRotFloats / 2 / kThreads;  // per thread, always read
    const float* rowrot = reinterpret_cast<const float*>(blob + layout_rowrot_offset(d.n_layers * d.n_kv)) +
                          static_cast<size_t>(layer * d.n_kv + kvh) * kRowRotFloats;
    // the query element of thread tid (clamped: in bounds, surplus unused),
    // read as the aligned 32-bit word that holds it
    const size_t qi = (static_cast<size_t>(lz) * hqn + kvh * G) * kHeadDim + min(tid, G * kHeadDim - 1);
    const bool bf = d.in_dtype == 1;
    const uint32_t qw = *reinterpret_cast<const uint32_t*>(static_cast<const uint8_t*>(q) +
                                                           (bf ? (qi * 2) & ~static_cast<size_t>(3) : qi * 4));
    const uint32_t mw = reinterpret_cast<const uint32_t*>(M->dim)[tid & 31];
    const uint32_t cv = c16[min(tid, kCodebookEntries - 1)];
    float rv[kRotFirst];
#pragma unroll
    for (int u = 0; u < kRotFirst; ++u) rv[u] = rowrot[tid + u * kThreads];
    if (tid < G * kHeadDim) qn[tid] = __uint_as_float(bf ? ((qi & 1) ? qw & 0xFFFF0000u : qw << 16) : qw);
    if (tid < 32) dimw[tid] = mw;
    // (fewer threads than query coordinates: the rest in a second round)
    for (int i = tid + kThreads; i < G * kHeadDim; i += kThreads)
      qn[i] = ld_q(q, (static_cast<size_t>(lz) * hqn + kvh * G) * kHeadDim + i, d.in_dtype);
    if (tid < kCodebookEntries) cbs[tid] = static_cast<uint16_t>(cv);
#pragma unroll
    for (int u = 0; u < kRotFirst; ++u)
      if (tid + u * kThreads < rtot) rs[tid + u * kThreads] = rv[u];
    // rows whose blocks exceed half the slot (few, large groups)
    for (int i = tid + kRotFirst * kThreads; i < rtot; i += kThreads) rs[i] = rowrot[i];
  }
  __syncthreads();
  for (int e = tid; e < G * kHeadDim; e += kThreads)
    qg[e] = qn[(e >> 7) * kHeadDim + reinterpret_cast<const uint8_t*>(dimw)[e & 127]];
  __syncthreads();
  for (int e = tid; e < G * kHeadDim; e += kThreads) {
    // one rotated coordinate per thread and round: p = stream position, g its group
    const int h = e >> 7, p = e & 127;
    int dg = rdim[0], off = roff[0], p0 = rpos[0];
#pragma unroll
    for (int g = 1; g < kMaxGroups; ++g)
      if (p >= rpos[g]) {
        dg = rdim[g];
        off = roff[g];
        p0 = rpos[g];
      }
    const int j = p - p0;
    const float* rt = rs + off;  // Pi_dg transposed: rt[k dg + j] = Pi[j][k]
    const float* qq = qg + h * kHeadDim + p0;
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
    int k = 0;
    for (; k + 4 <= dg; k += 4) {
      a0 = fmaf(rt[k * dg + j], qq[k], a0);
      a1 = fmaf(rt[(k + 1) * dg + j], qq[k + 1], a1);
      a2 = fmaf(rt[(k + 2) * dg + j], qq[k + 2], a2);
      a3 = fmaf(rt[(k + 3) * dg + j], qq[k + 3], a3);
    }
    if (k < dg) {  // d_g is even: two terms left
      a0 = fmaf(rt[k * dg + j], qq[k], a0);
      a1 = fmaf(rt[(k + 1) * dg + j], qq[k + 1], a1);
    }
    // log2(e) folded in: logits come out in base-2 units for exp2
    qr[e] = ((a0 + a1) + (a2 + a3)) * (kLog2e / sqrtf(static_cast<float>(dg) * kHeadDim));
  }
  __syncthreads();
  // ---- query image: slot s, lane 4b+i holds step 16(s - slot0_g) + b of
  // group g, head i of each set, 4 coordinates, as fp16 hi and lo parts.
  // Slots are numbered group after group; one pass over all of them.
  {
    int sl0[kMaxGroups], nslots = 0;
#pragma unroll
    for (int g = 0; g < kMaxGroups; ++g) {
      sl0[g] = nslots;
      nslots += ((rdim[g] + 3) / 4 + 15) / 16;
    }
    for (int i = tid; i < nslots * NSET * 64 * 4; i += kThreads) {
      const int k = i & 3, l = (i >> 2) & 63, set = (i >> 8) % NSET, slot = (i >> 8) / NSET;
      int gd = rdim[0], gp = rpos[0], s0 = sl0[0];
#pragma unroll
      for (int g = 1; g < kMaxGroups; ++g)
        if (g < ng && slot >= sl0[g]) {
          gd = rdim[g];
          gp = rpos[g];
          s0 = sl0[g];
        }
      const int step = 16 * (slot - s0) + (l >> 2), qh = 4 * set + (l & 3), coord = 4 * step + k;
      float v = 0.f;
      if (coord < gd && qh < G) v = qr[qh * kHeadDim + gp + coord];
      const _Float16 hi = static_cast<_Float16>(v);
      const _Float16 lo = static_cast<_Float16>(v - static_cast<float>(hi));
      uint8_t* dst = smem + kQimg + (((slot * 2 + set) * 2) * 64 + l) * 8 + k * 2;
      *reinterpret_cast<_Float16*>(dst) = hi;
      *reinterpret_cast<_Float16*>(dst + 64 * 8) = lo;
    }
  }
  __syncthreads();
  // ---- lookup tables
#pragma unroll
  for (int i = tid; i < 16 * 16; i += kThreads) {
    const int e = i >> 4;
    const uint16_t* cb = cbs + cb_index(1);
    *reinterpret_cast<uint2*>(smem + kLut1 + i * 8) =
        make_uint2(cb[e & 1] | (static_cast<uint32_t>(cb[(e >> 1) & 1]) << 16),
                   cb[(e >> 2) & 1] | (static_cast<uint32_t>(cb[(e >> 3) & 1]) << 16));
  }
  if constexpr (T12) {
    // 3-bit codes four at a time, in the byte table's place: entry i holds
    // the centroids of codes i & 7, (i >> 3) & 7, (i >> 6) & 7 and i >> 9
    // (one copy; 1-bit key codes then take the 4-code table)
    const uint16_t* cb = cbs + cb_index(3);
    for (int i = tid; i < 4096; i += kThreads)
      *reinterpret_cast<uint2*>(smem + kLut1B + i * 8) =
          make_uint2(cb[i & 7] | (static_cast<uint32_t>(cb[(i >> 3) & 7]) << 16),
                     cb[(i >> 6) & 7] | (static_cast<uint32_t>(cb[i >> 9]) << 16));
  } else {
#pragma unroll
    for (int i = tid; i < 256 * 8; i += kThreads) {
      const int e = i >> 3;  // code byte: bit c is the code of coordinate c
      const uint16_t* cb = cbs + cb_index(1);
      const auto pair = [&](int c) { return cb[(e >> c) & 1] | (static_cast<uint32_t>(cb[(e >> (c + 1)) & 1]) << 16); };
      *reinterpret_cast<uint4*>(smem + kLut1B + i * 16) = make_uint4(pair(0), pair(2), pair(4), pair(6));
    }
  }
#pragma unroll
  for (int i = tid; i < 256 * 32; i += kThreads) {
    const int e = i >> 5;
    const uint16_t* cb = cbs + cb_index(2);
    *reinterpret_cast<uint2*>(smem + kLut2 + i * 8) =
        make_uint2(cb[e & 3] | (static_cast<uint32_t>(cb[(e >> 2) & 3]) << 16),
                   cb[(e >> 4) & 3] | (static_cast<uint32_t>(cb[(e >> 6) & 3]) << 16));
  }
#pragma unroll
  for (int i = tid; i < 64 * 32; i += kThreads) {
    const int e = i >> 5;
    const uint16_t* cb = cbs + cb_index(3);
    *reinterpret_cast<uint32_t*>(smem + kLut3 + i * 4) = cb[e & 7] | (static_cast<uint32_t>(cb[(e >> 3) & 7]) << 16);
  }
#pragma unroll
  for (int i = tid; i < 256 * 8; i += kThreads) {
    const int e = i >> 3;
    const uint16_t* cb = cbs + cb_index(4);
    *reinterpret_cast<uint32_t*>(smem + kLut4 + i * 4) = cb[e & 15] | (static_cast<uint32_t>(cb[e >> 4]) << 16);
  }
#pragma unroll
  for (int i = tid; i < 32 * 32; i += kThreads)
    *reinterpret_cast<uint32_t*>(smem + kLut5 + i * 4) = cbs[cb_index(5) + (i >> 5)];
#pragma unroll
  for (int i = tid; i < 256 + 128 + 64; i += kThreads) {
    const int b = i < 256 ? 8 : (i < 384 ? 7 : 6);
    const int k = i < 256 ? i : (i < 384 ? i - 256 : i - 384);
    *reinterpret_cast<uint16_t*>(smem + kLutF + i * 2) = cbs[cb_index(b) + k];
  }
  __syncthreads();

  uint32_t gmb[8];
  LaneRep rep{static_cast<uint32_t>(kLut1 + (lane & 15) * 8), static_cast<uint32_t>(kLut3 + (lane & 31) * 4),
                    static_cast<uint32_t>(kLut4 + (lane & 7) * 4),   static_cast<uint32_t>(kLut5 + (lane & 31) * 4),
                    static_cast<uint32_t>(kLut2 + (lane & 31) * 8),  static_cast<uint32_t>(kLut1B + (T12 ? 0 : (lane & 7) * 16)),
                    static_cast<uint32_t>(kQimg + lane * 8)};
  // opaque to the compiler: with the bits of the bases unknown, a lookup
  // address stays (shifted field & mask) | base, one and-or
  asm volatile("" : "+v"(rep.r1), "+v"(rep.r3), "+v"(rep.r4), "+v"(rep.r5), "+v"(rep.r2), "+v"(rep.r1b));

  // a context length outside [0, max_ctx] (the host's bound, which sized
  // the splits) makes the sequence's outputs NaN instead of dropping rows
  const int ctx_raw = ctx_len[seq];
  const bool ctx_ok = ctx_raw >= 0 && ctx_raw <= d.max_ctx;
  const int ctx = min(ctx_raw, cap);
  // packed rows [t_lo, t_hi): all of them, or those between the protected
  // window's sink and recent rows (none when the window covers the context;
  // t_lo < 64, so the first tile of a non-empty range holds a row of it)
  int t_lo = 0, t_hi = ctx;
  if (win.part != nullptr) {
    const int ns = min(win.n_sink, ctx);
    t_lo = ns;
    t_hi = ctx - min(win.n_recent, ctx - ns);
    if (t_hi <= t_lo) t_lo = t_hi = 0;
  }
  const int t_begin = split * split_len;
  const int t_end = min(t_begin + split_len, t_hi);
  const size_t row = (static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + kvh;

  float m_run[NSET], l_run[NSET];
  float4_t O[NSET][2];
#pragma unroll
  for (int s = 0; s < NSET; ++s) {
    m_run[s] = kNegInf;
    l_run[s] = 0.f;
    O[s][0] = float4_t{0.f, 0.f, 0.f, 0.f};
    O[s][1] = float4_t{0.f, 0.f, 0.f, 0.f};
  }

  // Each wave walks its 64-token tiles with the next tile's keys in flight
  // while the current one is computed.
  const int stride = kWaves * 64;
  int t0 = t_begin + wave * 64;
  const int nslot = (ng + 1) & ~1;  // radius slots per token
  const RowPtrs R{c.k_codes + row * cap * kw, c.k_norms + row * kMaxGroups * cap,
                  c.v_codes + row * (cap / kTile) * kHeadDim * BV, c.v_norms + row * cap};
  // The next tile's keys are in flight while a tile is computed.  Its values
  // are too where the registers allow (one query set, rows of <= 8 words,
  // b_V <= 2);
  // otherwise a tile's values are loaded when it starts and used after its
  // QK products.
  constexpr bool kValuesAhead = NSET == 1 && KWB <= 8 && BV <= 2;
  uint32_t rw[KWB + kRowPad], knp[4], rw2[KWB], knp2[4], vw[4][pv_words<BV>()];
  uint32_t vw2[kValuesAhead ? 4 : 1][kValuesAhead ? pv_words<BV>() : 1];
  uint2 vn, vn2;
#pragma unroll
  for (int i = KWB; i < KWB + kRowPad; ++i) rw[i] = 0u;
  if (t0 < t_end) {
    load_keys<KWB>(rw2, knp2, nslot, R, kw, t0, lane);
    if constexpr (kValuesAhead) load_values<BV>(vn2, vw2, R, t0, lane);
  }
  for (; t0 < t_end; t0 += stride) {
#pragma unroll
    for (int i = 0; i < KWB; ++i) rw[i] = rw2[i];
#pragma unroll
    for (int p = 0; p < 4; ++p) knp[p] = knp2[p];
    if constexpr (kValuesAhead) {
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int w = 0; w < pv_words<BV>(); ++w) vw[p][w] = vw2[p][w];
      vn = vn2;
    } else {
      load_values<BV>(vn, vw, R, t0, lane);
    }
    // Wave priorities (the SIMD's issue arbiter prefers the higher one among
    // its waves): issuing the next tile's loads 3, QK products 2, PV products
    // 1, softmax 0, so that loads leave early and a wave in its softmax
    // (transcendentals and cross-lane steps) yields to the product phases
    // (-4.5 % time in A/B runs against no priorities)
    if (t0 + stride < t_end) {
      __builtin_amdgcn_s_setprio(3);
      load_keys<KWB>(rw2, knp2, nslot, R, kw, t0 + stride, lane);
      if constexpr (kValuesAhead) load_values<BV>(vn2, vw2, R, t0 + stride, lane);
      __builtin_amdgcn_s_setprio(0);
    }
    const int tk = t0 + lane;
    {
      // Re-read the row's width table every tile (scalar loads through an
      // opaque offset): hoisted out of the loop, its derived scalars exhaust
      // the SGPRs.
      uint32_t goff = 0;
      asm volatile("" : "+s"(goff));
      const uint32_t* gmt = reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint8_t*>(M->gm) + goff);
#pragma unroll
      for (int b = 0; b < 8; ++b) gmb[b] = gmt[b];
    }

    // ---------------- QK, one same-rate group at a time (lane = token)
    float4_t L[NSET];
#pragma unroll
    for (int s = 0; s < NSET; ++s) L[s] = float4_t{0.f, 0.f, 0.f, 0.f};
    __builtin_amdgcn_s_setprio(2);
    qk_all<NSET, T12, KWB>(std::make_integer_sequence<int, 8>{}, smem, rw, knp, gmb, rep, lane, L);
    __builtin_amdgcn_s_setprio(0);

    // ---------------- online softmax (lane 4b+i: head i, tokens 4b..4b+3)
    // Logits are in base-2 units (log2 e is folded into the query).  Only a
    // tile that reaches past the split end masks anything: its scores past
    // the end become -inf and their value radii 0.
    const bool full = t0 >= t_lo && t0 + 64 <= t_end;
    // value radii stay packed fp16: p n_V is one mixed-precision product
    // into each half of the PV operand (the codes' 1/sqrt(d_h) scales the
    // output instead)
    uint2 vr = vn;
    if (!full) {
      const int b0 = t0 + 4 * bq;  // radii of tokens outside [t_lo, t_end) are cleared
      const auto keep = [&](int j) { return b0 + j >= t_lo && b0 + j < t_end; };
      vr.x &= (keep(0) ? 0xFFFFu : 0u) | (keep(1) ? 0xFFFF0000u : 0u);
      vr.y &= (keep(2) ? 0xFFFFu : 0u) | (keep(3) ? 0xFFFF0000u : 0u);
    }
    half4_t pp[NSET];
#pragma unroll
    for (int s = 0; s < NSET; ++s) {
      float4_t x = L[s];
      if (!full) {
        if (tk >= t_end || tk < t_lo) x = float4_t{kNegInf, kNegInf, kNegInf, kNegInf};
        // (kept a branch: full tiles, nearly all of them, skip the selects)
        asm volatile("" : "+v"(x));
      }
      quad_transpose(x, lane);
      const float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
      // Most tiles raise no running maximum (one wave-wide vote on this
      // lane's four scores): the cross-lane maximum, the correction (exactly
      // 1) and the rescale are then skipped, which changes no result.
      float mn = m_run[s], corr = 1.f;
      const bool raise = __builtin_amdgcn_ballot_w64(mx > mn) != 0;
      if (raise) {
        mn = fmaxf(mn, xmax16(mx));
        corr = m_run[s] == kNegInf ? 0.f : exp2_hw(m_run[s] - mn);
      }
      float p[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) p[r] = exp2_hw(x[r] - mn);
      const float ps = ((p[0] + p[1]) + p[2]) + p[3];
      pp[s] = as_half4(mix_pair(p[0], p[1], vr.x), mix_pair(p[2], p[3], vr.y));
      l_run[s] = fmaf(l_run[s], corr, ps);  // this lane's tokens only; reduced after the loop
      if (raise) {
        const float c0 = qperm<0x00>(corr), c1 = qperm<0x55>(corr), c2 = qperm<0xAA>(corr), c3 = qperm<0xFF>(corr);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          O[s][h][0] *= c0;
          O[s][h][1] *= c1;
          O[s][h][2] *= c2;
          O[s][h][3] *= c3;
        }
        m_run[s] = mn;
      }
    }

    // ---------------- PV: 16 steps of 4 tokens (lane = dim)
    __builtin_amdgcn_s_setprio(1);
    pv_steps<BV, NSET, T12>(std::make_integer_sequence<int, 16>{}, smem, vw, rep, pp, O);
    __builtin_amdgcn_s_setprio(0);
  }

  finish_unit<NSET, kWaves>(smem, reinterpret_cast<int*>(smem + kGmeta), d, G, lz, kvh, split, tid, lane, wave,
                            m_run, l_run, O, counters, part, n_splits,
                            ctx_ok ? 0.08838834764831845f /* 1/sqrt(d_h) */ : opaque_nan(),
                            reinterpret_cast<const float*>(blob + kOffRotV), out, win.part);
}

// ---------------------------------------------------------------- fp16 comparator
// The same split-context decode over an uncompressed fp16 cache (keys and
// values [rows][128]): the same MFMA products, softmax and merges, with no
// decode and no rotation.  It is bound by HBM reads, so its workgroups are 4
// waves, one per SIMD: each wave has the SIMD's 512 registers (VGPRs and
// AGPRs) and keeps the next 64-row tile in flight while it computes the
// current one (about 300 registers; with two waves per SIMD, 256 each, the
// same schedule spills):
//  * keys: lane = token reads its 256-byte row with 16 loads of 16 bytes (two
//    4-coordinate steps each), the B operand of QK as it arrives;
//  * values: for each 4-token step and half of the dims, lane 4b + j reads 8
//    bytes (dims 64 h + 4b .. +3 of token 4s + j); a 4x4 transpose of 16-bit
//    elements inside each lane quad turns that into the PV B operand (4 tokens
//    of dim 64 h + lane).  32 loads per tile instead of 128 two-byte gathers.
// The next tile's keys are issued before the current QK products, its values
// right after them (into the registers the keys leave).
constexpr int kF16Waves = 4;
constexpr int kF16Threads = kF16Waves * 64;
constexpr int kF16Flag = (kF16Waves * 8 * 2 + kF16Waves * 8 * kHeadDim + 2 * 8 * kHeadDim) * 4;  // past the merge area
constexpr int kF16Lds = kF16Flag + 16;

template <int NSET, int S0, int... J>
__device__ __forceinline__ void f16_qk_chunk(std::integer_sequence<int, J...>, const uint4* ka,
                                             const half4_t (&qh)[NSET], const half4_t (&ql)[NSET],
                                             float4_t (&L)[NSET]) {
  (qk_mac<NSET, (S0 + J) % 16>((J & 1) ? as_half4(ka[J >> 1].z, ka[J >> 1].w) : as_half4(ka[J >> 1].x, ka[J >> 1].y),
                               qh, ql, L),
   ...);
}

// Keys of the tile at t0: lane = token, 16-byte chunks J0 .. J0 + 7 of its row.
template <int J0>
__device__ __forceinline__ void f16_load_keys(const _Float16* kb, int t0, int lane, uint4 (&k)[16]) {
  const uint4* kr = reinterpret_cast<const uint4*>(kb + static_cast<size_t>(t0 + lane) * kHeadDim);
#pragma unroll
  for (int j = J0; j < J0 + 8; ++j) k[j] = kr[j];
}
// Values of steps S0 .. S0 + 7 of the tile at t0, untransposed: v[2 s + h] =
// dims 64 h + 4 (lane / 4) .. +3 of token t0 + 4 s + lane % 4.
template <int S0>
__device__ __forceinline__ void f16_load_values(const _Float16* vb, int t0, int lane, uint2 (&v)[32]) {
  const _Float16* base = vb + static_cast<size_t>(t0 + (lane & 3)) * kHeadDim + 4 * (lane >> 2);
#pragma unroll
  for (int s = S0; s < S0 + 8; ++s)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      v[2 * s + h] = *reinterpret_cast<const uint2*>(base + static_cast<size_t>(4 * s) * kHeadDim + 64 * h);
}

// 4x4 transpose of 16-bit elements inside a lane quad: on entry lane j holds
// row j (elements 0, 1 in .x, 2, 3 in .y); on exit column j (rows 0, 1 in .x,
// 2, 3 in .y).  First 32-bit words move between lanes j and j ^ 2, then
// 16-bit halves between j and j ^ 1 (byte selects per lane parity).
struct QuadT16 {
  bool hi2;
  uint32_t sel_s, sel_0, sel_1;
};
__device__ __forceinline__ QuadT16 quad_t16_setup(int lane) {
  const bool odd = lane & 1;
  return QuadT16{(lane & 2) != 0, odd ? 0x05040100u : 0x07060302u, odd ? 0x03020504u : 0x05040100u,
                 odd ? 0x03020706u : 0x07060100u};
}
__device__ __forceinline__ half4_t quad_t16(uint2 w, const QuadT16& t) {
  const uint32_t x = t.hi2 ? w.x : w.y;
  const uint32_t y = static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0x4E, 0xF, 0xF, false));
  const uint32_t a = t.hi2 ? y : w.x;  // rows j & 1,       columns 2 (j >> 1) .. +1
  const uint32_t c = t.hi2 ? w.y : y;  // rows (j & 1) + 2, the same columns
  const uint32_t snd = __builtin_amdgcn_perm(c, a, t.sel_s);
  const uint32_t r = static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(snd), 0xB1, 0xF, 0xF, false));
  return as_half4(__builtin_amdgcn_perm(r, a, t.sel_0), __builtin_amdgcn_perm(r, c, t.sel_1));
}

// PV of step S (lane = dim): the step's values transposed in the lane quads
// (with MASK, rows past the split end zeroed first: the cache there may hold
// anything), then one MFMA per half of the dims and query set.
template <int NSET, bool MASK, int S>
__device__ __forceinline__ void f16_pv_step(const uint2 (&vc)[32], const QuadT16& qt, int lane, int t0, int t_end,
                                            const half4_t (&pp)[NSET], float4_t (&O)[NSET][2]) {
  // before the transpose lane 4b + j holds token 4 S + j of its dims
  const bool dead = MASK && t0 + 4 * S + (lane & 3) >= t_end;
  half4_t vv[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    uint2 w = vc[2 * S + h];
    if (MASK) w = dead ? make_uint2(0u, 0u) : w;
    vv[h] = quad_t16(w, qt);
  }
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int q = 0; q < NSET; ++q)
      O[q][h] = __builtin_amdgcn_mfma_f32_4x4x4f16(pp[q], vv[h], O[q][h], 4, S % 16, 0);
}
template <int NSET, bool MASK, int S0, int... J>
__device__ __forceinline__ void f16_pv(std::integer_sequence<int, J...>, const uint2 (&vc)[32], const QuadT16& qt,
                                       int lane, int t0, int t_end, const half4_t (&pp)[NSET],
                                       float4_t (&O)[NSET][2]) {
  (f16_pv_step<NSET, MASK, S0 + J>(vc, qt, lane, t0, t_end, pp, O), ...);
}
// PV of a whole tile; the values of the next tile's second half are issued
// between the two halves.
template <int NSET, bool MASK>
__device__ __forceinline__ void f16_pv_tile(const _Float16* vb, int tn, const uint2 (&vc)[32], uint2 (&vn)[32],
                                            const QuadT16& qt, int lane, int t0, int t_end,
                                            const half4_t (&pp)[NSET], float4_t (&O)[NSET][2]) {
  f16_pv<NSET, MASK, 0>(std::make_integer_sequence<int, 8>{}, vc, qt, lane, t0, t_end, pp, O);
  __builtin_amdgcn_sched_barrier(0);
  f16_load_values<8>(vb, tn, lane, vn);
  __builtin_amdgcn_sched_barrier(0);
  f16_pv<NSET, MASK, 8>(std::make_integer_sequence<int, 8>{}, vc, qt, lane, t0, t_end, pp, O);
}

// One 64-row tile at t0 (keys in kc, values in vc), with the loads of the tile
// at tn issued into kn and vn, each half as soon as the registers it replaces
// in the other set are consumed.
template <int NSET>
__device__ __forceinline__ void f16_tile(const uint8_t* smem, const _Float16* kb, const _Float16* vb, int t0, int tn,
                                         int t_end, int lane, uint32_t qlane, const QuadT16& qt, uint4 (&kc)[16],
                                         uint2 (&vc)[32], uint4 (&kn)[16], uint2 (&vn)[32], float (&m_run)[NSET],
                                         float (&l_run)[NSET], float4_t (&O)[NSET][2]) {
  // sched_barrier(0) keeps each prefetch between the products it was placed
  // after and before: hoisted further, the loads would hold registers that
  // the current tile still needs
  __builtin_amdgcn_s_setprio(2);
  f16_load_keys<0>(kb, tn, lane, kn);
  __builtin_amdgcn_sched_barrier(0);

  // ---------------- QK (lane = token), 32 steps
  float4_t L[NSET];
#pragma unroll
  for (int s = 0; s < NSET; ++s) L[s] = float4_t{0.f, 0.f, 0.f, 0.f};
  half4_t qh[NSET], ql[NSET];
#pragma unroll
  for (int slot = 0; slot < 2; ++slot) {
#pragma unroll
    for (int s = 0; s < NSET; ++s) {
      const uint32_t base = qlane + ((slot * 2 + s) * 2) * 64 * 8;
      const uint2 uh = lds64(smem, base), ul = lds64(smem, base + 64 * 8);
      qh[s] = as_half4(uh.x, uh.y);
      ql[s] = as_half4(ul.x, ul.y);
    }
    f16_qk_chunk<NSET, 0>(std::make_integer_sequence<int, 8>{}, kc + 8 * slot, qh, ql, L);
    f16_qk_chunk<NSET, 8>(std::make_integer_sequence<int, 8>{}, kc + 8 * slot + 4, qh, ql, L);
    __builtin_amdgcn_sched_barrier(0);
    if (slot == 0) f16_load_keys<8>(kb, tn, lane, kn);
    __builtin_amdgcn_sched_barrier(0);
  }
  f16_load_values<0>(vb, tn, lane, vn);
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_setprio(0);

  // ---------------- online softmax, as in the packed decode
  const bool full = t0 + 64 <= t_end;
  const int tk = t0 + lane;
  half4_t pp[NSET];
#pragma unroll
  for (int s = 0; s < NSET; ++s) {
    float4_t x = L[s];
    if (!full && tk >= t_end) x = float4_t{kNegInf, kNegInf, kNegInf, kNegInf};
    quad_transpose(x, lane);
    float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
    mx = xmax16(mx);
    const float mn = fmaxf(m_run[s], mx);
    const float corr = m_run[s] == kNegInf ? 0.f : exp2_hw(m_run[s] - mn);
    float ps = 0.f;
    half4_t ph;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float p = exp2_hw(x[r] - mn);
      ps += p;
      ph[r] = static_cast<_Float16>(p);
    }
    pp[s] = ph;
    l_run[s] = l_run[s] * corr + ps;
    if (__builtin_amdgcn_ballot_w64(mn != m_run[s]) != 0) {
      const float c0 = qperm<0x00>(corr), c1 = qperm<0x55>(corr), c2 = qperm<0xAA>(corr), c3 = qperm<0xFF>(corr);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        O[s][h][0] *= c0;
        O[s][h][1] *= c1;
        O[s][h][2] *= c2;
        O[s][h][3] *= c3;
      }
    }
    m_run[s] = mn;
  }

  // ---------------- PV (lane = dim), 16 steps of 4 tokens
  __builtin_amdgcn_s_setprio(1);
  if (full) f16_pv_tile<NSET, false>(vb, tn, vc, vn, qt, lane, t0, t_end, pp, O);
  else f16_pv_tile<NSET, true>(vb, tn, vc, vn, qt, lane, t0, t_end, pp, O);
  __builtin_amdgcn_s_setprio(0);
}

template <int NSET>
__global__ __launch_bounds__(kF16Threads) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_f16_mfma(Dims d, const void* __restrict__ q,
                                                          const int32_t* __restrict__ ctx_len,
                                                          const _Float16* __restrict__ k16,
                                                          const _Float16* __restrict__ v16, float* __restrict__ out,
                                                          int32_t* __restrict__ counters, float* __restrict__ part,
                                                          int n_splits, int split_len) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kF16Lds];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int item = static_cast<int>(__builtin_amdgcn_workgroup_id_x());
  const int split = item % n_splits, rest = item / n_splits;
  const int kvh = rest % d.n_kv, lz = rest / d.n_kv;
  const int layer = d.layer >= 0 ? d.layer : lz / d.batch;
  const int seq = lz % d.batch;
  const int G = d.group, hqn = d.n_kv * G, cap = d.capacity;

  // query image, 2 slots of 16 steps (as in the packed decode), logits in
  // base-2 units: q / sqrt(d_h) * log2 e, fp16 hi and lo parts
  static_assert(2 * 2 * 2 * 64 * 8 <= kF16Flag, "query image inside the merge area");
  for (int i = tid; i < 2 * NSET * 64 * 4; i += kF16Threads) {
    const int k = i & 3, l = (i >> 2) & 63, set = (i >> 8) % NSET, slot = (i >> 8) / NSET;
    const int step = 16 * slot + (l >> 2), qh = 4 * set + (l & 3), coord = 4 * step + k;
    float v = 0.f;
    if (qh < G)
      v = ld_q(q, (static_cast<size_t>(lz) * hqn + kvh * G + qh) * kHeadDim + coord, d.in_dtype) *
          (kLog2e / 11.313708498984761f);
    const _Float16 hi = static_cast<_Float16>(v);
    const _Float16 lo = static_cast<_Float16>(v - static_cast<float>(hi));
    uint8_t* dst = smem + (((slot * 2 + set) * 2) * 64 + l) * 8 + k * 2;
    *reinterpret_cast<_Float16*>(dst) = hi;
    *reinterpret_cast<_Float16*>(dst + 64 * 8) = lo;
  }
  __syncthreads();

  const int ctx_raw = ctx_len[seq];
  const bool ctx_ok = ctx_raw >= 0 && ctx_raw <= d.max_ctx;  // else NaN outputs, as in the packed decode
  const int ctx = min(ctx_raw, cap);
  const int t_begin = split * split_len;
  const int t_end = min(t_begin + split_len, ctx);
  const size_t row = (static_cast<size_t>(layer) * d.batch + seq) * d.n_kv + kvh;
  const _Float16* kb = k16 + row * cap * kHeadDim;
  const _Float16* vb = v16 + row * cap * kHeadDim;
  const uint32_t qlane = static_cast<uint32_t>(lane) * 8;
  const QuadT16 qt = quad_t16_setup(lane);

  float m_run[NSET], l_run[NSET];
  float4_t O[NSET][2];
#pragma unroll
  for (int s = 0; s < NSET; ++s) {
    m_run[s] = kNegInf;
    l_run[s] = 0.f;
    O[s][0] = O[s][1] = float4_t{0.f, 0.f, 0.f, 0.f};
  }
  // Every tile loaded lies below the capacity (a multiple of 64): a tile past
  // the split end (the prefetch after the last one, or a wave with no tile)
  // reloads the current tile or row 0 instead.
  constexpr int stride = kF16Waves * 64;
  int t0 = t_begin + wave * 64;
  uint4 kA[16], kB[16];
  uint2 vA[32], vB[32];
  {
    const int tl = t0 < t_end ? t0 : 0;
    f16_load_keys<0>(kb, tl, lane, kA);
    f16_load_keys<8>(kb, tl, lane, kA);
    f16_load_values<0>(vb, tl, lane, vA);
    f16_load_values<8>(vb, tl, lane, vA);
  }
  while (t0 < t_end) {
    int tn = t0 + stride < t_end ? t0 + stride : t0;
    f16_tile<NSET>(smem, kb, vb, t0, tn, t_end, lane, qlane, qt, kA, vA, kB, vB, m_run, l_run, O);
    t0 += stride;
    if (t0 >= t_end) break;
    tn = t0 + stride < t_end ? t0 + stride : t0;
    f16_tile<NSET>(smem, kb, vb, t0, tn, t_end, lane, qlane, qt, kB, vB, kA, vA, m_run, l_run, O);
    t0 += stride;
  }
  __syncthreads();
  finish_unit<NSET, kF16Waves>(smem, reinterpret_cast<int*>(smem + kF16Flag), d, G, lz, kvh, split, tid, lane,
                               wave, m_run, l_run, O, counters, part, n_splits, ctx_ok ? 1.f : opaque_nan(),
                               nullptr, out, nullptr);
}

inline hipError_t launch_f16_mfma_impl(const Dims& d, const void* q, const int32_t* ctx_len, const void* k16,
                                       const void* v16, float* out, const DecodeWs& ws, hipStream_t s) {
  dim3 grid(ws.n_splits * d.n_kv * d.batch * d.n_lc);
  const auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, dim3(kF16Threads), 0, s, d, q, ctx_len, static_cast<const _Float16*>(k16),
                       static_cast<const _Float16*>(v16), out, ws.counters, ws.part, ws.n_splits, ws.split_len);
  };
  if (d.group <= 4) go(k_f16_mfma<1>);
  else go(k_f16_mfma<2>);
  return hipGetLastError();
}

// Launch the packed decode for value width BV (one instantiation per file).
template <int BV>
hipError_t launch_split_bv_impl(const Dims& d, const void* layout, const void* q, const int32_t* ctx_len,
                                const CachePtrs& c, float* out, const DecodeWs& ws, hipStream_t s) {
  dim3 grid(ws.n_splits * d.n_kv * d.batch * d.n_lc);
  const uint8_t* blob = static_cast<const uint8_t*>(layout);
  const auto go = [&](auto kern, int threads) {
    hipLaunchKernelGGL(kern, grid, dim3(threads), 0, s, d, blob, q, ctx_len, c, out, ws.counters, ws.part,
                       ws.n_splits, ws.split_len, WinArgs{ws.wpart, ws.n_sink, ws.n_recent});
  };
  constexpr int t1 = split_waves<1>() * 64, t2 = split_waves<2>() * 64;
  if (d.group <= 4) {
    if (d.k_words <= 8) go(k_split_mfma<1, 8, BV>, t1);
    else if (d.k_words <= 12) go(k_split_mfma<1, 12, BV>, t1);
    else if (d.k_words <= 16) go(k_split_mfma<1, 16, BV>, t1);
    else go(k_split_mfma<1, 32, BV>, t1);
  } else {
    if (d.k_words <= 8) go(k_split_mfma<2, 8, BV>, t2);
    else if (d.k_words <= 12) go(k_split_mfma<2, 12, BV>, t2);
    else if (d.k_words <= 16) go(k_split_mfma<2, 16, BV>, t2);
    else go(k_split_mfma<2, 32, BV>, t2);
  }
  return hipGetLastError();
}

}  // namespace split_detail
}  // namespace bgtq
