// MFMA operand packing: K-major FP4 codes + scales -> "fragment-major" operands.
//
// Fragment (t, kb) of a [rows][K] operand covers rows 32t..32t+31 and K elements
// 64kb..64kb+63; lane l of the fragment holds row 32t + l%32 and the 32 K elements
// 64kb + 32(l/32) .. +31 exactly as the 32x32x64 scaled MFMA consumes them, so one wave
// loads a fragment as one contiguous block.  Rows past the end and the missing half of an
// MXFP4 half step are zero codes.
//
//   MXFP4 (A or B): 16 B per lane (E2M1 nibbles) + 1 B per lane (E8M0 scale).
//   HiF4 A (activations): 48 B per lane = E2M3 "hi" then "lo" (V = 16 hi + lo, see
//                         device_fp4.h) + 1 B per lane (the level-1 code c1).
//   HiF4 B (weights):     24 B per lane = BF6 E3M2 of k 2^-b + 1 B per lane (c1).
#include "kernels.h"
#include "device_fp4.h"

namespace resq {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ void put6(uint32_t* out, int i, uint32_t f) {
  const int bit = 6 * i;
  out[bit >> 5] |= f << (bit & 31);
  if ((bit & 31) > 26) out[(bit >> 5) + 1] |= f >> (32 - (bit & 31));
}

// Lane record l of K step kb of row tile t.
template <int MODE>
__device__ __forceinline__ void pack_record(const uint8_t* __restrict__ codes, const void* __restrict__ scales,
                                            int64_t rows, int64_t K, int64_t nkb, uint8_t* __restrict__ frag,
                                            uint8_t* __restrict__ fscale, int64_t t, int64_t kb, int l) {
  const int64_t gid = (t * nkb + kb) * 64 + l;
  const int64_t row = t * 32 + (l & 31);
  const int half = l >> 5;
  const bool in = row < rows && kb * 64 + half * 32 < K;
  uint4 cw = make_uint4(0, 0, 0, 0);
  if (in) cw = *reinterpret_cast<const uint4*>(codes + row * (K / 2) + kb * 32 + half * 16);
  if constexpr (MODE == kPackMx) {
    uint8_t sc = 0;
    if (in) sc = reinterpret_cast<const uint8_t*>(scales)[row * (K / 32) + kb * 2 + half];
    *reinterpret_cast<uint4*>(frag + gid * 16) = cw;
    fscale[gid] = sc;
  } else {
    uint32_t mt = 0;
    if (in) mt = reinterpret_cast<const uint32_t*>(scales)[row * (K / 64) + kb];
    const uint32_t c1 = mt & 0xFFu;
    const uint32_t words[4] = {cw.x, cw.y, cw.z, cw.w};
    uint32_t a[6] = {0, 0, 0, 0, 0, 0}, b[6] = {0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const uint32_t code = (words[i >> 3] >> (4 * (i & 7))) & 15u;
      const int h = half * 8 + (i >> 2);
      const int sh = (int)((mt >> (8 + (h >> 1))) & 1u) + (int)((mt >> (16 + h)) & 1u);
      if constexpr (MODE == kPackHiA) {
        uint32_t hi, lo;
        hif4_split_e2m3(code, (int)c1, sh, hi, lo);
        put6(a, i, hi);
        put6(b, i, lo);
      } else {
        put6(a, i, hif4_e3m2(code, sh));
      }
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

// grid: x covers the lane records of one row tile (64 per K step), y = row tiles (grid-stride)
template <int MODE>
__global__ __launch_bounds__(kThreads) void pack_kernel(const uint8_t* __restrict__ codes,
                                                        const void* __restrict__ scales,
                                                        int64_t rows, int64_t K, int64_t nfrag_rows,
                                                        uint8_t* __restrict__ frag,
                                                        uint8_t* __restrict__ fscale) {
  const int64_t nkb = (K + 63) / 64;
  const int64_t local = (int64_t)blockIdx.x * kThreads + threadIdx.x;  // kb * 64 + lane
  if (local >= nkb * 64) return;
  for (int64_t t = blockIdx.y; t < nfrag_rows; t += gridDim.y)
    pack_record<MODE>(codes, scales, rows, K, nkb, frag, fscale, t, local >> 6, (int)(local & 63));
}

}  // namespace

size_t frag_bytes(int mode, int64_t rows, int64_t K) {
  const int64_t n = ((rows + 31) / 32) * ((K + 63) / 64) * 64;
  const int64_t per = mode == kPackMx ? 16 : (mode == kPackHiA ? 48 : 24);
  return (size_t)(n * per);
}

size_t frag_scale_bytes(int64_t rows, int64_t K) {
  return (size_t)(((rows + 31) / 32) * ((K + 63) / 64) * 64);
}

void launch_pack(int mode, const uint8_t* codes, const void* scales, int64_t rows, int64_t K,
                 uint8_t* frag, uint8_t* fscale, hipStream_t s) {
  const int64_t nfr = (rows + 31) / 32, per_tile = ((K + 63) / 64) * 64;
  if (nfr == 0 || per_tile == 0) return;
  const dim3 grid((unsigned)((per_tile + kThreads - 1) / kThreads), (unsigned)(nfr < 65535 ? nfr : 65535));
  if (mode == kPackMx)
    hipLaunchKernelGGL((pack_kernel<kPackMx>), grid, dim3(kThreads), 0, s, codes, scales, rows, K, nfr, frag, fscale);
  else if (mode == kPackHiA)
    hipLaunchKernelGGL((pack_kernel<kPackHiA>), grid, dim3(kThreads), 0, s, codes, scales, rows, K, nfr, frag, fscale);
  else
    hipLaunchKernelGGL((pack_kernel<kPackHiB>), grid, dim3(kThreads), 0, s, codes, scales, rows, K, nfr, frag, fscale);
}

}  // namespace resq
