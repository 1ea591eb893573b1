// Device helpers shared by the fused, unfused and decode kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fqk {

typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef __bf16 bf16x2_t __attribute__((__vector_size__(2 * sizeof(__bf16))));
typedef float f32x4_t __attribute__((__vector_size__(4 * sizeof(float))));
typedef uint32_t u32x4_t __attribute__((__vector_size__(4 * sizeof(uint32_t))));

// ---------------------------------------------------------------------------
// INT4 -> bf16 MFMA operand.
//
// A 32-bit word of Wq holds the codes of 8 consecutive k of one column, code
// j in bits 4j..4j+3.  The bf16 value 128 + q has bit pattern 0x4300 | q
// (exponent 2^7, q in the low four mantissa bits, whose unit is 1), so one
// and-or turns the codes sitting in bits 0..3 and 16..19 of a word into a
// packed bf16 pair without any conversion instruction: the pairs come out as
// (k0,k4), (k1,k5), (k2,k6), (k3,k7) after shifts by 0, 4, 8 and 12.  The
// activation operand is staged in that same order, so the 8-term dot product
// the MFMA forms per lane is unchanged.  The offset 128 + z is removed after
// each 128-row group with the exact identity
//     sum_k x_k (q_k - z) = sum_k x_k (128 + q_k) - (128 + z) sum_k x_k,
// so (q - z) never needs to be formed and the scale s is applied in fp32 once
// per group (eq. 3 of the paper).  The fp32 sums are at most 143 sum|x_k|,
// which keeps their rounding error near 1e-6 of the result.
// ---------------------------------------------------------------------------
// (a & b) | c as one VALU operation (gfx950 three-input bitwise op; truth
// table 0xEA).  Plain C++ for this pattern compiles to two VOP2 operations,
// because a VOP3 encoding cannot carry the two literal constants.
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0xEA);
}

constexpr float kCodeOffset = 128.f;   // value of the bf16 bit pattern 0x4300

// Two words (two columns) at once, each into its 8-element operand: the
// and-or above on the word shifted by 0, 4, 8 and 12.  One 64-bit shift of
// the pair (w1:w0) yields w1 >> s in its high half and w0 >> s in its low
// half, polluted only in bits 32-s..31 by w1's low bits, which the nibble mask
// clears for s <= 12, so three 64-bit shifts replace six 32-bit ones (4.5
// against 2 x 3.1 cycles measured per instruction).
template <int S>
__device__ __forceinline__ uint64_t shr64c(uint64_t p) {
  uint64_t r;
  asm("v_lshrrev_b64 %0, %2, %1" : "=v"(r) : "v"(p), "i"(S));
  return r;
}

__device__ __forceinline__ void dequant_pair(uint32_t w0, uint32_t w1, bf16x8_t& b0, bf16x8_t& b1) {
  const uint32_t mask = 0x000F000Fu, bias = 0x43004300u;
  const uint64_t p = (uint64_t(w1) << 32) | w0;
  const uint64_t s4 = shr64c<4>(p), s8 = shr64c<8>(p), s12 = shr64c<12>(p);
  u32x4_t r0, r1;
  r0[0] = and_or(w0, mask, bias);
  r1[0] = and_or(w1, mask, bias);
  r0[1] = and_or(uint32_t(s4), mask, bias);
  r1[1] = and_or(uint32_t(s4 >> 32), mask, bias);
  r0[2] = and_or(uint32_t(s8), mask, bias);
  r1[2] = and_or(uint32_t(s8 >> 32), mask, bias);
  r0[3] = and_or(uint32_t(s12), mask, bias);
  r1[3] = and_or(uint32_t(s12 >> 32), mask, bias);
  b0 = __builtin_bit_cast(bf16x8_t, r0);
  b1 = __builtin_bit_cast(bf16x8_t, r1);
}

// Position of element k%8 inside an 8-element chunk of the LDS activation
// rows: chunk order is (x0, x4, x1, x5, x2, x6, x3, x7).
__device__ __forceinline__ uint32_t chunk_pos(uint32_t k) {
  return (k & ~7u) | ((k & 3u) << 1) | ((k >> 2) & 1u);
}

// Same map applied to four packed u8 row indices at once.
__device__ __forceinline__ uint32_t chunk_pos4(uint32_t k4) {
  return and_or(k4, 0xF8F8F8F8u, and_or(k4 << 1, 0x06060606u, (k4 >> 2) & 0x01010101u));
}

// 16 bytes of X (x0..x7) -> chunk order (x0,x4,x1,x5,x2,x6,x3,x7): one byte
// permute per output dword.
__device__ __forceinline__ uint4 permute_chunk(uint4 w) {
  uint4 o;
  o.x = __builtin_amdgcn_perm(w.z, w.x, 0x05040100u);   // x0 | x4 << 16
  o.y = __builtin_amdgcn_perm(w.z, w.x, 0x07060302u);   // x1 | x5 << 16
  o.z = __builtin_amdgcn_perm(w.w, w.y, 0x05040100u);   // x2 | x6 << 16
  o.w = __builtin_amdgcn_perm(w.w, w.y, 0x07060302u);   // x3 | x7 << 16
  return o;
}

// ---------------------------------------------------------------------------
// One Tile-COO group (16 bytes, four slots), decoded as the paper's outlier
// decoding step describes (Sec. 4.2): four u8 rows, four u8 columns, four
// bf16 values; value bits 0x0000 mark a padding slot.
// ---------------------------------------------------------------------------
struct Group {
  uint32_t rows;   // k0 | k1 << 8 | k2 << 16 | k3 << 24 (tile-local)
  uint32_t cols;   // n0 | n1 << 8 | n2 << 16 | n3 << 24 (tile-local)
  uint32_t v01;    // bf16 v0 | v1 << 16
  uint32_t v23;    // bf16 v2 | v3 << 16
};

__device__ __forceinline__ Group decode_group(uint4 g) {
  Group d;
  d.rows = g.x;
  d.cols = g.y;
  d.v01 = g.z;
  d.v23 = g.w;
  return d;
}

__device__ __forceinline__ uint32_t slot_row(const Group& d, int j) { return (d.rows >> (8 * j)) & 0xFFu; }
__device__ __forceinline__ uint32_t slot_col(const Group& d, int j) { return (d.cols >> (8 * j)) & 0xFFu; }
__device__ __forceinline__ uint32_t slot_val(const Group& d, int j) {
  return ((j < 2 ? d.v01 : d.v23) >> (16 * (j & 1))) & 0xFFFFu;
}
// All four slots in one column (always true in by-column mode).
__device__ __forceinline__ bool single_column(const Group& d) {
  return d.cols == (d.cols & 0xFFu) * 0x01010101u;
}

// ---------------------------------------------------------------------------
// Number formats.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits) {
  return __builtin_bit_cast(float, bits << 16);
}

__device__ __forceinline__ float f16_bits_to_f32(uint32_t bits) {
  return float(__builtin_bit_cast(_Float16, uint16_t(bits)));
}

// fp32 -> bf16, round to nearest, ties to even (IEEE 754 rounding applied to
// the 16 dropped bits); NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return ((u >> 16) | 0x40u) & 0xFFFFu;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

}  // namespace fqk
