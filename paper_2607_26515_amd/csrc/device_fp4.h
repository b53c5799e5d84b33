// Device-side FP4 arithmetic for gfx950: MXFP4 and HiF4 block quantization and the
// operand encodings the scaled f8f6f4 MFMA consumes.
//
// Every decision (block scale, element code, level-2/3 bits) is exact: scales are read from
// the exponent and fraction fields of the block maximum, and element codes come from
// comparisons with thresholds that are small integers times powers of two (exact in float32),
// after a power-of-two rescale with v_ldexp_f32 (exact; fp32 denormals are kept).  No
// reciprocal or division is used, since HiF4 scales are not powers of two.  Inputs are finite.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace resq {

constexpr int kMxBlock = 32;
constexpr int kHiBlock = 64;

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// v from another lane of the same row of 16 through a DPP lane pattern (every pattern used
// reads inside the row; all lanes active).
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // lane i of 8 <- lane 7-i
constexpr int kDppMirror = 0x140;      // lane i of 16 <- lane 15-i

// Larger of two magnitudes (finite, +0 or positive): their bit patterns order as integers.
__device__ __forceinline__ float max_mag(float a, float b) {
  return __uint_as_float(max(__float_as_uint(a), __float_as_uint(b)));
}

// Max of a magnitude v (finite, +0 or positive) over aligned groups of G lanes (G a power of
// two <= 64).  Up to 16 lanes the partners come through DPP: after the maxima over lane pairs
// and quads, the mirrored lane of an 8-group lies in the other quad and that of a 16-group in
// the other 8-group.
template <int G>
__device__ __forceinline__ float group_max(float v) {
  uint32_t u = __float_as_uint(v);
  if constexpr (G >= 2) u = max(u, dpp_u32<kDppXor1>(u));
  if constexpr (G >= 4) u = max(u, dpp_u32<kDppXor2>(u));
  if constexpr (G >= 8) u = max(u, dpp_u32<kDppHalfMirror>(u));
  if constexpr (G >= 16) u = max(u, dpp_u32<kDppMirror>(u));
#pragma unroll
  for (int o = 16; o < G; o <<= 1) u = max(u, (uint32_t)__shfl_xor((int)u, o, 64));
  return __uint_as_float(u);
}

template <int G>
__device__ __forceinline__ double group_sum(double v) {
#pragma unroll
  for (int o = 1; o < G; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ------------------------------------------------------------------------------------------
// MXFP4: E2M1 elements, one E8M0 scale per 32 elements (OCP MX conversion rule, paper Sec. 3)
// ------------------------------------------------------------------------------------------
// Shared exponent of a block with max magnitude amax (finite, +0 or positive):
// floor(log2 amax) - 2, clamped to [-127, 127].  For normal amax that is the biased exponent
// field minus 129 (at most 125); a subnormal amax or zero has field 0 and clamps to -127.
__device__ __forceinline__ int mx_exponent(float amax) {
  const int e = (int)(__float_as_uint(amax) >> 23) - 129;
  return e < -127 ? -127 : e;
}

// 4-bit code of x under exponent E: nearest E2M1 magnitude, ties to the even code, saturating.
__device__ __forceinline__ uint32_t mx_code(float x, int E) {
  const float y = ldexpf(fabsf(x), -E);  // exact power-of-two rescale
  const uint32_t k = (y > 0.25f) + (y >= 0.75f) + (y > 1.25f) + (y >= 1.75f) + (y > 2.5f) +
                     (y >= 3.5f) + (y > 5.0f);
  return ((__float_as_uint(x) >> 28) & 8u) | k;
}

__device__ __forceinline__ float e2m1_mag(uint32_t k) {
  // {0, .5, 1, 1.5, 2, 3, 4, 6}
  const float lo = (float)(k & 1) * 0.5f + (float)((k >> 1) & 1) * 1.0f;  // k<4: k/2
  if (k < 4) return lo;
  return (k == 4) ? 2.f : (k == 5) ? 3.f : (k == 6) ? 4.f : 6.f;
}

__device__ __forceinline__ float mx_value(uint32_t code, int E) {
  const float v = ldexpf(e2m1_mag(code & 7), E);
  return (code & 8) ? -v : v;
}

// 2^E as a float for the MX exponent range E in [-127, 127] (2^-127 is subnormal).
__device__ __forceinline__ float mx_scale_f32(int E) {
  return E >= -126 ? __uint_as_float((uint32_t)(E + 127) << 23) : __uint_as_float(0x00400000u);
}

// The same quantization on gfx950's scaled conversions, two elements per instruction:
// v_cvt_scalef32_pk_fp4_f32 with scale 2^E rounds x / 2^E to the nearest E2M1 magnitude,
// ties to the even code, saturates at 6 and keeps the sign of a zero result, which is
// mx_code's definition; v_cvt_scalef32_pk_f32_fp4 returns mx_value.  (GPU tests compare the
// resulting codes and scales with the oracle's on every E2M1 tie and threshold, saturation,
// signed zeros and shared exponents from -127, where 2^E is subnormal, to 124.)
// Codes of x0, x1: bits 0-3 and 4-7 of the result.
__device__ __forceinline__ uint32_t mx_code2(float x0, float x1, float scale) {
  return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, x0, x1, scale, 0) & 0xFFu;
}
__device__ __forceinline__ void mx_value2(uint32_t codes2, float scale, float& v0, float& v1) {
  const auto v = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(codes2, scale, 0);
  v0 = v[0];
  v1 = v[1];
}

// ------------------------------------------------------------------------------------------
// HiF4 (reading stated in resq.h): 64-element blocks, E6M2 level-1 scale, one-bit level-2
// (per 8) and level-3 (per 4) down-shifts, S1P2 elements k/4.
//   s1 = 2^(e-31) (1 + m/4) for code c = 4e + m;  element value = k (4+m) 2^(e-35-b)
// ------------------------------------------------------------------------------------------
// Smallest code c with 1.75 * s1(c) >= A (saturating at 255), for a magnitude A (finite, +0 or
// positive).  For A in [2^ea, 2^(ea+1)) the values 1.75 * s1 of codes 4(ea+30)+1 .. +4 are
// {35, 42, 49, 56, 63} 2^(ea-5), i.e. mantissas 1.09375, 1.3125, 1.53125, 1.75 and above 1.875,
// so c is that base code plus the number of the first four that A's mantissa exceeds, read
// straight from its exponent and fraction fields.  Subnormal A (ea < -126) and every A below
// 2^-31 give a negative count, clamped to code 0.
__device__ __forceinline__ int hif4_c1(float A) {
  const uint32_t u = __float_as_uint(A);
  const int E = (int)(u >> 23);  // biased exponent ea + 127
  const uint32_t f = u & 0x7FFFFFu;
  const int c = 4 * E - 387 + (f > 0x0C0000u) + (f > 0x280000u) + (f > 0x440000u) + (f > 0x600000u);
  return c < 0 ? 0 : (c > 255 ? 255 : c);
}

// 1.75 * s1 / 2 * 2^-shift = 7 (4+m) 2^(e-36-shift): the "fits at half the scale" threshold.
__device__ __forceinline__ float hif4_half_fit(int c1, int shift) {
  return ldexpf((float)(7 * (4 + (c1 & 3))), (c1 >> 2) - 36 - shift);
}

// The midpoints of the element grid of level-1 code c1 that hif4_k compares with, in units of
// 2^(e-36-b): q, 3q, 7q and 11q, and the step 2q (q = 4+m; small integers, exact).
struct Hif4Mid {
  float q, q2, q3, q7, q11;
};
__device__ __forceinline__ Hif4Mid hif4_mid(int c1) {
  const float q = (float)(4 + (c1 & 3));
  Hif4Mid t{q, 2.f * q, 3.f * q, 7.f * q, 11.f * q};
  // Kept opaque: the optimiser would otherwise turn the per-element choice between 3q and 11q
  // into an integer multiply and a conversion.
  asm("" : "+v"(t.q3), "+v"(t.q11));
  return t;
}

// Magnitude k (0..7) of |x| on the grid k/4 * s, s = s1 2^-b: nearest, ties to even k.
// On the rescaled y = |x| 2^(36+b-e) the midpoint between j and j+1 is (2j+1) q; a tie goes to
// the even neighbour, so y must exceed the midpoint above an even j and reach the one above an
// odd j.  k is the number of midpoints passed, found by a three-step binary search: 3|4 (7q),
// then 1|2 (3q) or 5|6 (11q), then the midpoint above the even k so far, 2q further up or
// down.  NaN passes none (k = 0), +inf all (k = 7).
__device__ __forceinline__ uint32_t hif4_k(float x, int c1, int b, const Hif4Mid& t) {
  const float y = ldexpf(fabsf(x), 36 + b - (c1 >> 2));
  const bool h4 = y >= t.q7;
  const float t2 = h4 ? t.q11 : t.q3;
  const bool h2 = y >= t2;
  const float t1 = t2 + (h2 ? t.q2 : -t.q2);
  const bool h1 = y > t1;
  return (h4 ? 4u : 0u) + (h2 ? 2u : 0u) + (h1 ? 1u : 0u);
}

__device__ __forceinline__ float hif4_value(uint32_t code, int c1, int b) {
  const float v = ldexpf((float)((code & 7) * (4 + (c1 & 3))), (c1 >> 2) - 35 - b);
  return (code & 8) ? -v : v;
}

// The grid step of level-1 code c1 and shift b, (4+m) 2^(e-35-b) (exact and normal: at least
// 4 * 2^-37), and the element value k * step carrying the sign of x, which is the code's sign
// (k = 0 included: a signed zero); k * step <= 7 * 7 * 2^28 is exact.  The quantizers use this
// form: one conversion, one multiply and one sign insertion per element.
__device__ __forceinline__ float hif4_step(int c1, int b) {
  return ldexpf((float)(4 + (c1 & 3)), (c1 >> 2) - 35 - b);
}
__device__ __forceinline__ float hif4_signed_value(uint32_t k, float step, float x) {
  return copysignf((float)k * step, x);
}

// Compress the even bits of a 16-bit value into 8 bits.
__device__ __forceinline__ uint32_t even_bits16(uint32_t x) {
  x &= 0x5555u;
  x = (x | (x >> 1)) & 0x3333u;
  x = (x | (x >> 2)) & 0x0F0Fu;
  x = (x | (x >> 4)) & 0x00FFu;
  return x;
}

// ------------------------------------------------------------------------------------------
// MFMA operand encodings for HiF4 (f8f6f4 MFMA, formats: 2 = FP6 E2M3, 3 = BF6 E3M2)
// ------------------------------------------------------------------------------------------
// Activation side: V = k (4+m) 2^(2-b) <= 196 (value = V 2^(e-37)) is split V = 16 hi + lo;
// hi, lo <= 15 are E2M3 codes of hi/8, lo/8 (E2M3 code t has value t/8 for t <= 15), each
// with the element's sign in bit 5.  Scales: hi term 2^(e-30) -> E8M0 e + 97, lo term
// 2^(e-34) -> E8M0 e + 93.
// hif4_split4 splits the four elements of one level-3 group (shift b) at once: their codes in
// the low nibbles of the bytes of nb (high nibbles ignored), q2 = 4+m in both 16-bit lanes.
// One 16-bit-lane multiply forms the four products k (4+m) <= 49 (no carry crosses a byte)
// and one shift applies 2 - b (V <= 196 stays in its byte); the four 6-bit hi and lo fields
// then close up into 24 bits each, field j at bit 6j.
__device__ __forceinline__ uint32_t close_up6x4(uint32_t x) {  // bytes f0..f3 (< 64) -> 24 bits
  const uint32_t t = (x & 0x003F003Fu) | ((x >> 2) & 0x0FC00FC0u);
  return (t & 0xFFFu) | ((t >> 4) & 0xFFF000u);
}
__device__ __forceinline__ void hif4_split4(uint32_t nb, uint32_t q2, uint32_t b, uint32_t& hi24, uint32_t& lo24) {
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  const uint32_t k = nb & 0x07070707u, sg = (nb & 0x08080808u) << 2;
  const uint32_t kq = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, k) * __builtin_bit_cast(u16x2, q2));
  const uint32_t V = kq << (2u - b);
  hi24 = close_up6x4(sg | ((V >> 4) & 0x0F0F0F0Fu));
  lo24 = close_up6x4(sg | (V & 0x0F0F0F0Fu));
}

// Weight side: k 2^-b as a BF6 E3M2 code (value exact), sign in bit 5; the remaining
// factor (4+m) 2^(e-35) is the E8M0 scale e + 92 times the per-column factor (4+m).  The
// E3M2 code (bias 3) of k = 0..7 is 0, 12 (1.0), 16 (2.0), 18 (3.0), 20, 21, 22, 23, and the
// shift b lowers the exponent field of a nonzero one by b.
// hif4_e3m2x4 encodes the four elements of one level-3 group (shift b) at once, their codes
// in the low nibbles of the bytes of nb (high nibbles ignored): the codes of k come from a
// byte table by v_perm, nonzero ones lowered by b << 2 (at least 12 - 8, so no borrow crosses
// a byte), the sign goes to bit 5, and the four 6-bit fields close up into 24 bits, field j
// at bit 6j.
__device__ __forceinline__ uint32_t hif4_e3m2x4(uint32_t nb, uint32_t b) {
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  const uint32_t k = nb & 0x07070707u;
  const uint32_t e = __builtin_amdgcn_perm(0x17161514u, 0x12100C00u, k);  // 0 12 16 18 20 21 22 23
  const uint32_t nz = ((k + 0x7F7F7F7Fu) & 0x80808080u) >> 7;              // 1 in each nonzero byte
  const uint32_t sub = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, nz) *
                                                        __builtin_bit_cast(u16x2, (4u * b) * 0x00010001u));
  return close_up6x4(((nb & 0x08080808u) << 2) | (e - sub));
}

}  // namespace resq
