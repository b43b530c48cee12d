// Device helpers shared by the TwinQuant HIP kernels (gfx950 / MI355X).
//
// Numeric conventions (paper Sec. 2 Eq. 1, Sec. 4.3):
//  * a group's scale is s = fp16_rne(fp32(max|v|) / 7) (IEEE fp32 division);
//  * a code is q = clamp(rint(fp32(v) / s), -7, 7), 0 when s == 0;
//  * codes reach the matrix cores as fp8 e4m3 bytes whose exponent field is
//    zero: byte = sign << 7 | |q| encodes q * 2^-9 exactly (e4m3 subnormals),
//    so every product is exact and a 64-term dot product of codes, with both
//    operand block scales set to 2^9, comes out of the fp32 accumulator as the
//    exact integer sum.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tq {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kGroup = 64;
constexpr int kScale2p9 = 127 + 9;  // E8M0 block scale 2^9

// TQ4 word -> two words of fp8 e4m3 bytes (codes 0..3 and 4..7, in order).
__device__ __forceinline__ void tq4_to_fp8(uint32_t w, uint32_t &lo, uint32_t &hi) {
  lo = w & 0x87878787u;
  hi = __builtin_amdgcn_alignbit(w, w, 4) & 0x87878787u;
}

// 32 codes (4 TQ4 words, natural order) -> one fp8 matrix-core operand.
__device__ __forceinline__ v8i unpack32(u32x4 raw) {
  v8i r;
  uint32_t lo, hi;
  tq4_to_fp8(raw.x, lo, hi); r[0] = (int)lo; r[1] = (int)hi;
  tq4_to_fp8(raw.y, lo, hi); r[2] = (int)lo; r[3] = (int)hi;
  tq4_to_fp8(raw.z, lo, hi); r[4] = (int)lo; r[5] = (int)hi;
  tq4_to_fp8(raw.w, lo, hi); r[6] = (int)lo; r[7] = (int)hi;
  return r;
}

// Eight codes in [-7, 7] -> one TQ4 word.
__device__ __forceinline__ uint32_t tq4_pack8(const int c[8]) {
  uint32_t w = 0;
#pragma unroll
  for (int i = 0; i < 4; i++) {
    uint32_t m = (uint32_t)(c[i] < 0 ? -c[i] : c[i]);
    w |= m << (8 * i);
    w |= (uint32_t)(c[i] < 0) << (8 * i + 7);
    uint32_t m2 = (uint32_t)(c[4 + i] < 0 ? -c[4 + i] : c[4 + i]);
    w |= m2 << (8 * i + 4);
    w |= (uint32_t)(c[4 + i] < 0) << (8 * ((i + 1) & 3) + 3);
  }
  return w;
}

// fp8 byte of a code (sign-magnitude e4m3 subnormal).
__device__ __forceinline__ uint32_t code_to_fp8(int q) {
  return (uint32_t)(q < 0 ? (0x80 | -q) : q);
}

__device__ __forceinline__ float half_bits_to_float(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}

__device__ __forceinline__ uint16_t float_to_half_bits(float f) {
  return __builtin_bit_cast(uint16_t, (_Float16)f);  // v_cvt_f16_f32, round to nearest even
}

__device__ __forceinline__ float bf16_bits_to_float(uint16_t b) {
  return __builtin_bit_cast(float, (uint32_t)b << 16);
}

__device__ __forceinline__ uint16_t float_to_bf16_bits(float f) {
  uint32_t b = __builtin_bit_cast(uint32_t, f);
  b += 0x7fffu + ((b >> 16) & 1u);  // round to nearest even (finite inputs)
  return (uint16_t)(b >> 16);
}

// Scale of a group from its max |v|: fp16(max / 7) and its fp32 value.
__device__ __forceinline__ float q4_scale(float amax, uint16_t &s16) {
  float s32 = amax / 7.0f;  // IEEE division (no fast-math anywhere in this library)
  s16 = float_to_half_bits(s32);
  return half_bits_to_float(s16);
}

__device__ __forceinline__ int q4_code(float v, float s) {
  if (s == 0.0f) return 0;
  float t = __builtin_rintf(v / s);
  t = t > 7.0f ? 7.0f : (t < -7.0f ? -7.0f : t);
  return (int)t;
}

// Exact integer dot products of 32x32 code tiles over one group of 64:
// D[i][j] = sum_k A[i][k] * B[k][j].  Operand lane l holds row/column l % 32,
// k in [32 * (l / 32), +32); result lane l holds column l % 32, rows
// 8 * (v / 4) + 4 * (l / 32) + v % 4 for v = 0..15.
__device__ __forceinline__ v16f mfma_codes_32x32x64(v8i a, v8i b) {
  const v16f z = {0};
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, z, 0, 0, 0, kScale2p9, 0, kScale2p9);
}
// the same added to c (exact while the sums stay integers below 2^24)
__device__ __forceinline__ v16f mfma_codes_32x32x64_acc(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, kScale2p9, 0, kScale2p9);
}

// Same for 16x16 tiles over 128 k: operand lane l holds row/column l % 16,
// k in [32 * (l / 16), +32); result lane l: column l % 16, rows 4 * (l / 16) + v.
__device__ __forceinline__ v4f mfma_codes_16x16x128(v8i a, v8i b) {
  const v4f z = {0};
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, z, 0, 0, 0, kScale2p9, 0, kScale2p9);
}

// Activation quantizer step shared by the quantizer kernel and the decode
// kernel's fp16 entry: eight lanes own one 64-value group, eight values each.
// max over the 8 lanes 8 j .. 8 j + 7 with DPP lane swizzles: swap neighbours,
// swap pairs, then mirror the two quads of the eight
__device__ __forceinline__ float max8_dpp(float a) {
  a = fmaxf(a, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), 0xB1, 0xF, 0xF, false)));
  a = fmaxf(a, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), 0x4E, 0xF, 0xF, false)));
  a = fmaxf(a, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), 0x141, 0xF, 0xF, false)));
  return a;
}

// Codes of eight fp16 values v of one group with fp16 scale s (s > 0, or 0
// for a group that quantizes to zeros), as fp8 operand bytes: lo holds codes
// 0..3, hi codes 4..7.  y is 1 / s to within a few ulp (0 when s == 0).
//
// For fp16 v and s the exact quotient v / s is either a half-integer or at
// least 2.4e-4 away from every half-integer (write v = A 2^p, s = B 2^q with
// |A|, B < 2^11: a non-zero distance is a multiple of 2^(min(p+1, q) - q) /
// (2B)), so rounding t = v * y to the nearest integer already gives
// rint(v / s) except on exact ties.  A tie shows in the exact remainder
// r = v - rint(t) s (one fma; the product and the difference are exact in
// fp32) as |r| = s / 2, and round-half-to-even then takes 2 rint(t / 2), the
// even one of the two neighbours (t / 2 lies within rounding error of an odd
// multiple of 1/4, far from any rounding boundary).  This is the remainder
// correction of Markstein's division method, specialised to a quotient needed
// only to the nearest integer.  The clamped code q becomes the byte
// sign << 7 | |q| as the e4m3 value q 2^-9 (a subnormal, converted exactly;
// the fma adds +0 so a zero code is never -0).
__device__ __forceinline__ void quant8_fp8(const float (&v)[8], float s, float y, uint32_t &lo,
                                           uint32_t &hi) {
  const float hs = 0.5f * s;
  float f[8];
#pragma unroll
  for (int e = 0; e < 8; e++) {
    const float t = v[e] * y;
    const float q = __builtin_rintf(t);
    const float r = fmaf(-q, s, v[e]);
    const float qe = 2.0f * __builtin_rintf(0.5f * t);
    const float c = fminf(fmaxf(fabsf(r) == hs ? qe : q, -7.0f), 7.0f);
    f[e] = fmaf(c, 0x1p-9f, 0.0f);
  }
  lo = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(f[0], f[1], 0, false);
  lo = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(f[2], f[3], (int)lo, true);
  hi = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(f[4], f[5], 0, false);
  hi = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(f[6], f[7], (int)hi, true);
}

__device__ __forceinline__ int row_of_32x32(int lane, int v) {
  return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}

}  // namespace tq
