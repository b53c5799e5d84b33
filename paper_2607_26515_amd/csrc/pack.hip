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
#include "frag.h"

namespace resq {
namespace {

constexpr int kThreads = 256;

// Lane record l of K step kb of row tile t.  MASK: 0 none; 1 kept channels (bit j of gbits
// = column j); 2 kept 32 x 64 blocks (bit I * (K / 64) + J of gbits).  Pruned elements
// become the +0 code.
template <int MODE, int MASK>
__device__ __forceinline__ void pack_record(const uint8_t* __restrict__ codes, const void* __restrict__ scales,
                                            int64_t rows, int64_t K, int64_t nkb, const uint8_t* __restrict__ gbits,
                                            uint8_t* __restrict__ frag, uint8_t* __restrict__ fscale, int64_t t,
                                            int64_t kb, int l) {
  const int64_t gid = (t * nkb + kb) * 64 + l;
  const int64_t row = t * 32 + (l & 31);
  const int half = l >> 5;
  const int64_t col = kb * 64 + half * 32;
  const bool in = row < rows && col < K;
  uint4 cw = make_uint4(0, 0, 0, 0);
  uint32_t sc = 0;
  if (in) {
    cw = *reinterpret_cast<const uint4*>(codes + row * (K / 2) + col / 2);
    if constexpr (MODE == kPackMx) sc = reinterpret_cast<const uint8_t*>(scales)[row * (K / 32) + col / 32];
    else sc = reinterpret_cast<const uint32_t*>(scales)[row * (K / 64) + kb];
    if constexpr (MASK == 1) {
      const uint32_t keep = *reinterpret_cast<const uint32_t*>(gbits + col / 8);  // 32 columns
      cw.x &= nibble_mask8(keep & 0xFFu);
      cw.y &= nibble_mask8((keep >> 8) & 0xFFu);
      cw.z &= nibble_mask8((keep >> 16) & 0xFFu);
      cw.w &= nibble_mask8(keep >> 24);
    } else if constexpr (MASK == 2) {
      const int64_t bit = (row / 32) * (K / 64) + kb;
      if (!((gbits[bit >> 3] >> (bit & 7)) & 1u)) cw = make_uint4(0, 0, 0, 0);
    }
  }
  store_frag_record<MODE>(frag, fscale, gid, cw, sc, half);
}

// grid: x covers the lane records of one row tile (64 per K step), y = row tiles (grid-stride)
template <int MODE, int MASK>
__global__ __launch_bounds__(kThreads) void pack_kernel(const uint8_t* __restrict__ codes,
                                                        const void* __restrict__ scales,
                                                        int64_t rows, int64_t K, int64_t nfrag_rows,
                                                        const uint8_t* __restrict__ gbits,
                                                        uint8_t* __restrict__ frag,
                                                        uint8_t* __restrict__ fscale) {
  const int64_t nkb = (K + 63) / 64;
  const int64_t local = (int64_t)blockIdx.x * kThreads + threadIdx.x;  // kb * 64 + lane
  if (local >= nkb * 64) return;
  for (int64_t t = blockIdx.y; t < nfrag_rows; t += gridDim.y)
    pack_record<MODE, MASK>(codes, scales, rows, K, nkb, gbits, frag, fscale, t, local >> 6, (int)(local & 63));
}

// Zero fill of n floats (grid-stride).
__global__ __launch_bounds__(kThreads) void zero_f32_kernel(float* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads)
    p[i] = 0.f;
}

}  // namespace

void launch_zero_f32(float* p, int64_t n, hipStream_t s) {
  if (n <= 0) return;
  const int64_t blocks = (n + kThreads - 1) / kThreads;
  hipLaunchKernelGGL(zero_f32_kernel, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(kThreads), 0, s, p, n);
}

size_t frag_bytes(int mode, int64_t rows, int64_t K) {
  const int64_t n = ((rows + 31) / 32) * ((K + 63) / 64) * 64;
  const int64_t per = mode == kPackMx ? 16 : (mode == kPackHiA ? 48 : 24);
  return (size_t)(n * per);
}

size_t frag_scale_bytes(int64_t rows, int64_t K) {
  return (size_t)(((rows + 31) / 32) * ((K + 63) / 64) * 64);
}

void launch_pack(int mode, const uint8_t* codes, const void* scales, int64_t rows, int64_t K,
                 uint8_t* frag, uint8_t* fscale, hipStream_t s, int mask, const uint8_t* gbits) {
  const int64_t nfr = (rows + 31) / 32, per_tile = ((K + 63) / 64) * 64;
  if (nfr == 0 || per_tile == 0) return;
  const dim3 grid((unsigned)((per_tile + kThreads - 1) / kThreads), (unsigned)(nfr < 65535 ? nfr : 65535));
#define RESQ_PK(M, K_) hipLaunchKernelGGL((pack_kernel<M, K_>), grid, dim3(kThreads), 0, s, codes, scales, rows, K, nfr, gbits, frag, fscale)
#define RESQ_PK_MASK(M) \
  if (mask == 1) RESQ_PK(M, 1); else if (mask == 2) RESQ_PK(M, 2); else RESQ_PK(M, 0);
  if (mode == kPackMx) { RESQ_PK_MASK(kPackMx) }
  else if (mode == kPackHiA) { RESQ_PK_MASK(kPackHiA) }
  else RESQ_PK(kPackHiB, 0);
#undef RESQ_PK_MASK
#undef RESQ_PK
}

}  // namespace resq
