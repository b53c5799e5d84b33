// Cooperative quantization of one block-scaled FP4 block, four elements per lane.
//
// A lane owns 4 consecutive elements along the block axis.  An MXFP4 block (32 elements)
// spans 8 aligned lanes, a HiF4 block (64) spans 16, a HiF4 level-2 group (8) spans 2 and a
// level-3 group (4) is one lane.  All lanes of a block must be active.
#pragma once

#include "device_fp4.h"

namespace resq {

enum Fmt { kMX = 0, kHI = 1 };

struct Quad {
  uint32_t code[4];  // 4-bit codes (sign << 3 | magnitude)
  float val[4];      // dequantized values (exact in float32)
  uint32_t scale;    // MX: E8M0 byte; HiF4: metadata word (same on every lane of the block)
  int c1;            // HiF4 level-1 code
  int b;             // HiF4 level-2 + level-3 shift of this lane's 4 elements
  int E;             // MX shared exponent
};

template <int FMT>
__device__ __forceinline__ Quad quantize_quad(const float x[4]) {
  Quad q;
  float a = fmaxf(fmaxf(fabsf(x[0]), fabsf(x[1])), fmaxf(fabsf(x[2]), fabsf(x[3])));
  if constexpr (FMT == kMX) {
    const float amax = group_max<8>(a);
    q.E = mx_exponent(amax);
    q.scale = (uint32_t)(q.E + 127);
    q.c1 = 0;
    q.b = 0;
    const float sc = mx_scale_f32(q.E);
#pragma unroll
    for (int i = 0; i < 4; i += 2) {
      const uint32_t c2 = mx_code2(x[i], x[i + 1], sc);
      q.code[i] = c2 & 15u;
      q.code[i + 1] = c2 >> 4;
      mx_value2(c2, sc, q.val[i], q.val[i + 1]);
    }
  } else {
    const float A = group_max<16>(a);
    q.c1 = hif4_c1(A);
    const float ag = max_mag(a, __uint_as_float(dpp_u32<kDppXor1>(__float_as_uint(a))));
    const int b2 = ag <= hif4_half_fit(q.c1, 0) ? 1 : 0;
    const int b3 = a <= hif4_half_fit(q.c1, b2) ? 1 : 0;
    q.b = b2 + b3;
    q.E = 0;
    const int lane = __lane_id();
    const int base = lane & ~15;
    const uint64_t m3 = __ballot(b3);
    const uint64_t m2 = __ballot(b2 && ((lane & 1) == 0));
    const uint32_t bits3 = (uint32_t)(m3 >> base) & 0xFFFFu;
    const uint32_t bits2 = even_bits16((uint32_t)(m2 >> base) & 0xFFFFu);
    q.scale = (uint32_t)q.c1 | (bits2 << 8) | (bits3 << 16);
    const Hif4Mid mid = hif4_mid(q.c1);
    const float step = hif4_step(q.c1, q.b);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t k = hif4_k(x[i], q.c1, q.b, mid);
      q.code[i] = ((__float_as_uint(x[i]) >> 28) & 8u) | k;
      q.val[i] = hif4_signed_value(k, step, x[i]);
    }
  }
  return q;
}

__device__ __forceinline__ uint32_t pack_quad_codes(const uint32_t c[4]) {
  return c[0] | (c[1] << 4) | (c[2] << 8) | (c[3] << 12);
}

// S_2:4 on one group of four: keep the two largest magnitudes, lower index on ties.
// Magnitude codes are monotone in |value| within a block (shared scale), so codes compare.
// Key i = magnitude << 2 | (3 - i) is distinct per element and orders by magnitude, then by
// lower index; the kept pair are the keys at or above the second largest.
__device__ __forceinline__ uint32_t keep_2_of_4(const uint32_t c[4]) {
  uint32_t k[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) k[i] = ((c[i] & 7u) << 2) | (uint32_t)(3 - i);
  const uint32_t hi01 = max(k[0], k[1]), lo01 = min(k[0], k[1]);
  const uint32_t hi23 = max(k[2], k[3]), lo23 = min(k[2], k[3]);
  const uint32_t second = max(min(hi01, hi23), max(lo01, lo23));
  uint32_t keep = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) keep |= (k[i] >= second ? 1u : 0u) << i;
  return keep;
}

// S_k:g on one group of G (4 or 8) consecutive elements given as magnitudes on one common
// grid: keep the k largest, lower index on ties.  Key i = mag << 3 | (G - 1 - i) is distinct per
// element and orders by magnitude, then by lower index; element i is kept when fewer than k
// keys exceed its own.
template <int G>
__device__ __forceinline__ uint32_t keep_k_of_g(const uint32_t mag[G], int k) {
  uint32_t key[G];
#pragma unroll
  for (int i = 0; i < G; ++i) key[i] = (mag[i] << 3) | (uint32_t)(G - 1 - i);
  uint32_t keep = 0;
#pragma unroll
  for (int i = 0; i < G; ++i) {
    int above = 0;
#pragma unroll
    for (int j = 0; j < G; ++j) above += (j != i && key[j] > key[i]) ? 1 : 0;
    keep |= (above < k ? 1u : 0u) << i;
  }
  return keep;
}

// The keep bits of the local pattern S_k:G for 8 consecutive codes (two groups when G = 4;
// S_2:4 itself takes keep_2_of_4).
// b[h] is the HiF4 level-2 + level-3 shift of elements 4h .. 4h+3 (0 for MXFP4, whose 8
// aligned elements share one scale).  A 4-group shares its scale, so its codes compare
// directly; an 8-group spans two HiF4 level-3 groups, so each magnitude code k is put on the
// finer common grid as k << (2 - b) (value = k/4 * s1 * 2^-b).
template <int G>
__device__ __forceinline__ uint32_t keep_local8(const uint32_t c[8], const int b[2], int k) {
  if constexpr (G == 8) {
    uint32_t mag[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) mag[i] = (c[i] & 7u) << (2 - b[i / 4]);
    return keep_k_of_g<8>(mag, k);
  } else {
    const uint32_t a[4] = {c[0], c[1], c[2], c[3]}, e[4] = {c[4], c[5], c[6], c[7]};
    uint32_t ma[4], me[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ma[i] = a[i] & 7u;
      me[i] = e[i] & 7u;
    }
    return keep_k_of_g<4>(ma, k) | (keep_k_of_g<4>(me, k) << 4);
  }
}

}  // namespace resq
