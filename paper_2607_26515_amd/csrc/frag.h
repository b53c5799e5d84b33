// One lane record of a fragment-major MFMA operand (layout in pack.hip): the 32 K-major codes
// (one uint4, element 2i in the low nibble of byte i) of row 32t + l%32, K elements
// 64kb + 32(l/32) .. +31, and their scale word (MX: the E8M0 byte; HiF4: the metadata word
// of the 64-block), written as record `gid` of `frag` plus its scale byte in `fscale`.
#pragma once

#include "device_fp4.h"
#include "kernels.h"

namespace resq {

// The HiF4 activation split (hif4_split4) of a 32-element lane record: field i of the record
// at bit 6i of hi (a) and lo (b).
__device__ __forceinline__ void hif4_split_record(const uint32_t words[4], uint32_t scale, int half,
                                                  uint32_t a[6], uint32_t b[6]) {
  const uint32_t q2 = (4u + (scale & 3u)) * 0x00010001u;
  const uint32_t l2 = scale >> (8 + 4 * half), l3 = scale >> (16 + 8 * half);
  uint32_t ch[8], cl[8];
#pragma unroll
  for (int g = 0; g < 8; ++g) {
    const uint32_t w = words[g >> 1];
    const uint32_t t = __builtin_amdgcn_perm(w, w, (g & 1) ? 0x0C030C02u : 0x0C010C00u);
    // nibble 4(g&1)+j of w in the low nibble of byte j (the high nibbles are ignored)
    hif4_split4(t | (t << 4), q2, ((l2 >> (g >> 1)) & 1u) + ((l3 >> g) & 1u), ch[g], cl[g]);
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    a[3 * h] = ch[4 * h] | (ch[4 * h + 1] << 24);
    a[3 * h + 1] = (ch[4 * h + 1] >> 8) | (ch[4 * h + 2] << 16);
    a[3 * h + 2] = (ch[4 * h + 2] >> 16) | (ch[4 * h + 3] << 8);
    b[3 * h] = cl[4 * h] | (cl[4 * h + 1] << 24);
    b[3 * h + 1] = (cl[4 * h + 1] >> 8) | (cl[4 * h + 2] << 16);
    b[3 * h + 2] = (cl[4 * h + 2] >> 16) | (cl[4 * h + 3] << 8);
  }
}

// Nibble mask keeping the elements whose bit is set in `keep` (bit e = element e of a word).
__device__ __forceinline__ uint32_t nibble_mask8(uint32_t keep) {
  uint32_t m = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) m |= ((keep >> e) & 1u) * (0xFu << (4 * e));
  return m;
}

// half = l / 32 (which 32-element half of the 64-element HiF4 block the record holds).
template <int MODE>
__device__ __forceinline__ void store_frag_record(uint8_t* __restrict__ frag, uint8_t* __restrict__ fscale,
                                                  int64_t gid, uint4 cw, uint32_t scale, int half) {
  if constexpr (MODE == kPackMx) {
    *reinterpret_cast<uint4*>(frag + gid * 16) = cw;
    fscale[gid] = (uint8_t)scale;
  } else {
    const uint32_t c1 = scale & 0xFFu;
    const uint32_t words[4] = {cw.x, cw.y, cw.z, cw.w};
    uint32_t a[6] = {0, 0, 0, 0, 0, 0}, b[6] = {0, 0, 0, 0, 0, 0};
    if constexpr (MODE == kPackHiA) {
      hif4_split_record(words, scale, half, a, b);
    } else {
      const uint32_t l2 = scale >> (8 + 4 * half), l3 = scale >> (16 + 8 * half);
      uint32_t c[8];
#pragma unroll
      for (int g = 0; g < 8; ++g) {
        const uint32_t w = words[g >> 1];
        const uint32_t t = __builtin_amdgcn_perm(w, w, (g & 1) ? 0x0C030C02u : 0x0C010C00u);
        c[g] = hif4_e3m2x4(t | (t << 4), ((l2 >> (g >> 1)) & 1u) + ((l3 >> g) & 1u));
      }
      a[0] = c[0] | (c[1] << 24);
      a[1] = (c[1] >> 8) | (c[2] << 16);
      a[2] = (c[2] >> 16) | (c[3] << 8);
      a[3] = c[4] | (c[5] << 24);
      a[4] = (c[5] >> 8) | (c[6] << 16);
      a[5] = (c[6] >> 16) | (c[7] << 8);
    }
    if constexpr (MODE == kPackHiA) {
      uint4* p = reinterpret_cast<uint4*>(frag + gid * 48);
      p[0] = make_uint4(a[0], a[1], a[2], a[3]);
      p[1] = make_uint4(a[4], a[5], b[0], b[1]);
      p[2] = make_uint4(b[2], b[3], b[4], b[5]);
    } else {
      uint2* p = reinterpret_cast<uint2*>(frag + gid * 24);
      p[0] = make_uint2(a[0], a[1]);
      p[1] = make_uint2(a[2], a[3]);
      p[2] = make_uint2(a[4], a[5]);
    }
    fscale[gid] = (uint8_t)c1;
  }
}

}  // namespace resq
