// Quantization passes: Q along rows or columns, the fused residual pass of the ResQ linear
// (Q(X), dX = X - Q(X), Q(dX), S_2:4) and the HiF4 MFMA operand packing.
#include "kernels.h"
#include "quant_core.h"

namespace resq {
namespace {

constexpr int kThreads = 256;

template <bool F32>
__device__ __forceinline__ float load1(const void* x, int64_t i) {
  if constexpr (F32) return reinterpret_cast<const float*>(x)[i];
  else return bf16_to_f32(reinterpret_cast<const uint16_t*>(x)[i]);
}

// 4 consecutive elements; VEC = the address is 8-byte (bf16) / 16-byte (f32) aligned.
template <bool F32, bool VEC>
__device__ __forceinline__ void load4(const void* x, int64_t i, float v[4]) {
  if constexpr (VEC && F32) {
    const float4 t = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(x) + i);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else if constexpr (VEC) {
    const uint2 t = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(x) + i);
    v[0] = bf16_to_f32(t.x & 0xFFFFu); v[1] = bf16_to_f32(t.x >> 16);
    v[2] = bf16_to_f32(t.y & 0xFFFFu); v[3] = bf16_to_f32(t.y >> 16);
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = load1<F32>(x, i + k);
  }
}

template <int FMT>
__device__ __forceinline__ void store_scale(void* scales, int64_t row, int64_t K, int64_t j4,
                                            uint32_t sc) {
  if constexpr (FMT == kMX) {
    if ((threadIdx.x & 7) == 0) reinterpret_cast<uint8_t*>(scales)[row * (K / 32) + j4 / 8] = (uint8_t)sc;
  } else {
    if ((threadIdx.x & 15) == 0) reinterpret_cast<uint32_t*>(scales)[row * (K / 64) + j4 / 16] = sc;
  }
}

// ---------------------------------------------------------------------------------------
// Q along rows: one lane per 4 elements, grid (ceil(cols/1024), rows)
// ---------------------------------------------------------------------------------------
template <int FMT, bool F32, bool VEC>
__global__ __launch_bounds__(kThreads) void quant_rows_kernel(const void* __restrict__ x,
                                                              int64_t rows, int64_t cols,
                                                              int64_t ld,
                                                              uint8_t* __restrict__ codes,
                                                              void* __restrict__ scales) {
  const int64_t j4 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (4 * j4 >= cols) return;  // whole blocks drop out together (cols % block == 0)
  for (int64_t row = blockIdx.y; row < rows; row += gridDim.y) {
    float v[4];
    load4<F32, VEC>(x, row * ld + 4 * j4, v);
    const Quad q = quantize_quad<FMT>(v);
    *reinterpret_cast<uint16_t*>(codes + row * (cols / 2) + 2 * j4) = (uint16_t)pack_quad_codes(q.code);
    store_scale<FMT>(scales, row, cols, j4, q.scale);
  }
}

// ---------------------------------------------------------------------------------------
// Q along columns (transposed output): 64 x 64 tiles staged through LDS
// ---------------------------------------------------------------------------------------
template <int FMT, bool F32>
__global__ __launch_bounds__(kThreads) void quant_cols_kernel(const void* __restrict__ x,
                                                              int64_t rows, int64_t cols,
                                                              int64_t ld,
                                                              uint8_t* __restrict__ codes,
                                                              void* __restrict__ scales) {
  __shared__ float tile[64][65];
  const int64_t r0 = (int64_t)blockIdx.y * 64;
  const int64_t c0 = (int64_t)blockIdx.x * 64;
  for (int i = threadIdx.x; i < 64 * 64; i += kThreads) {
    const int rr = i >> 6, cc = i & 63;
    float v = 0.f;
    if (r0 + rr < rows && c0 + cc < cols) v = load1<F32>(x, (r0 + rr) * ld + c0 + cc);
    tile[rr][cc] = v;
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int idx = it * kThreads + threadIdx.x;
    const int cc = idx >> 4, h = idx & 15;  // column, group of 4 rows
    float v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = tile[4 * h + k][cc];
    const Quad q = quantize_quad<FMT>(v);
    const int64_t col = c0 + cc;
    const int64_t j4 = r0 / 4 + h;  // position along K (= rows) in units of 4
    if (col < cols && 4 * j4 < rows) {
      *reinterpret_cast<uint16_t*>(codes + col * (rows / 2) + 2 * j4) = (uint16_t)pack_quad_codes(q.code);
      if constexpr (FMT == kMX) {
        if ((h & 7) == 0) reinterpret_cast<uint8_t*>(scales)[col * (rows / 32) + j4 / 8] = (uint8_t)q.scale;
      } else {
        if (h == 0) reinterpret_cast<uint32_t*>(scales)[col * (rows / 64) + j4 / 16] = q.scale;
      }
    }
  }
}

// ---------------------------------------------------------------------------------------
// Fragment-major output (see pack.hip): lane record of row `row`, K half of 64-block.
// ---------------------------------------------------------------------------------------
template <int FMT>
__device__ __forceinline__ void store_frag(uint8_t* __restrict__ frag, uint8_t* __restrict__ fsc,
                                           int64_t row, int64_t d, int64_t j4, const Quad& q,
                                           const uint32_t c[4]) {
  const int64_t nkb = (d + 63) / 64;
  const int64_t kb = j4 >> 4;      // 16 lanes of 4 elements per 64-block
  const int half = (int)((j4 >> 3) & 1);
  const int64_t f = ((row >> 5) * nkb + kb) * 64 + (row & 31) + 32 * half;
  if constexpr (FMT == kMX) {
    *reinterpret_cast<uint16_t*>(frag + f * 16 + (j4 & 7) * 2) = (uint16_t)pack_quad_codes(c);
    if ((j4 & 7) == 0) fsc[f] = (uint8_t)q.scale;
    if ((d & 63) != 0 && kb == nkb - 1) {
      // d % 64 == 32: the last K step has no second half; give it zero codes and a zero
      // scale byte (never the E8M0 NaN code)
      *reinterpret_cast<uint16_t*>(frag + (f + 32) * 16 + (j4 & 7) * 2) = 0;
      if ((j4 & 7) == 0) fsc[f + 32] = 0;
    }
  } else {
    // this lane's 4 elements as 24-bit E2M3 hi / lo runs; 8 lanes make one 48-byte record
    uint32_t h = 0, l = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      uint32_t hk, lk;
      hif4_split_e2m3(c[k], q.c1, q.b, hk, lk);
      h |= hk << (6 * k);
      l |= lk << (6 * k);
    }
    const int lane = __lane_id();
    const int base = lane & ~7, qi = lane & 7;
    const int qq = qi < 6 ? qi : 5;
    const int L = (32 * qq) / 24, o = 32 * qq - 24 * L;  // dword qq = bits [32qq, 32qq+32)
    const uint32_t h0 = __shfl(h, base + L, 64), h1 = __shfl(h, base + L + 1, 64);
    const uint32_t l0 = __shfl(l, base + L, 64), l1 = __shfl(l, base + L + 1, 64);
    if (qi < 6) {
      uint32_t* rec = reinterpret_cast<uint32_t*>(frag + f * 48);
      rec[qi] = (h0 >> o) | (h1 << (24 - o));
      rec[6 + qi] = (l0 >> o) | (l1 << (24 - o));
    }
    if (qi == 0) fsc[f] = (uint8_t)q.c1;
  }
}

// ---------------------------------------------------------------------------------------
// Residual pass of Eq. 2 / Eq. 4: Q(X), dX = X - Q(X) (float32, exact), Q(dX), S_2:4.
// FRAG: write MFMA fragments (rows m..m_rows-1 are zero padding of the last row tile)
// instead of K-major codes + scales.
// ---------------------------------------------------------------------------------------
template <int FMT, int MODE, bool VEC, bool FRAG>
__global__ __launch_bounds__(kThreads) void residual_kernel(
    const uint16_t* __restrict__ X, int64_t m, int64_t m_rows, int64_t d, int64_t ldx,
    uint8_t* __restrict__ qx_codes, void* __restrict__ qx_scales, uint8_t* __restrict__ qr_codes,
    void* __restrict__ qr_scales, uint8_t* __restrict__ keep_mask, double* __restrict__ partials) {
  const int64_t j4 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (4 * j4 >= d) return;
  for (int64_t row = blockIdx.y; row < m_rows; row += gridDim.y) {
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (row < m) load4<false, VEC>(X, row * ldx + 4 * j4, v);
    const Quad qx = quantize_quad<FMT>(v);
    if constexpr (FRAG) {
      store_frag<FMT>(qx_codes, reinterpret_cast<uint8_t*>(qx_scales), row, d, j4, qx, qx.code);
    } else {
      *reinterpret_cast<uint16_t*>(qx_codes + row * (d / 2) + 2 * j4) = (uint16_t)pack_quad_codes(qx.code);
      store_scale<FMT>(qx_scales, row, d, j4, qx.scale);
    }
    if constexpr (MODE != kResidNone) {
      float r[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) r[k] = v[k] - qx.val[k];  // exact in float32
      const Quad qr = quantize_quad<FMT>(r);
      uint32_t keep = 0xFu;
      if constexpr (MODE == kResid24) keep = keep_2_of_4(qr.code);
      uint32_t c[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) c[k] = ((keep >> k) & 1u) ? qr.code[k] : 0u;
      if constexpr (FRAG) {
        store_frag<FMT>(qr_codes, reinterpret_cast<uint8_t*>(qr_scales), row, d, j4, qr, c);
      } else {
        *reinterpret_cast<uint16_t*>(qr_codes + row * (d / 2) + 2 * j4) = (uint16_t)pack_quad_codes(c);
        store_scale<FMT>(qr_scales, row, d, j4, qr.scale);
        if (keep_mask != nullptr && MODE != kResidDense) {
          const uint32_t other = __shfl_xor(keep, 1, 64);
          if ((threadIdx.x & 1) == 0) keep_mask[row * (d / 8) + j4 / 2] = (uint8_t)(keep | (other << 4));
        }
        if (partials != nullptr) {
          // exact per-scale-block sum of squares (shared power-of-two factor, small integers)
          double sq = 0.0;
#pragma unroll
          for (int k = 0; k < 4; ++k) sq += (double)qr.val[k] * (double)qr.val[k];
          constexpr int G = (FMT == kMX) ? 8 : 16;
          sq = group_sum<G>(sq);
          if ((threadIdx.x & (G - 1)) == 0) partials[row * (d / (4 * G)) + j4 / G] = sq;
        }
      }
    }
  }
}

inline unsigned grid_rows(int64_t rows) { return (unsigned)(rows < 65535 ? rows : 65535); }

}  // namespace

void launch_quant_rows(int fmt, const void* x, bool in_f32, int64_t rows, int64_t cols,
                       int64_t ld, uint8_t* codes, void* scales, hipStream_t s) {
  if (rows == 0 || cols == 0) return;
  const dim3 grid((unsigned)((cols / 4 + kThreads - 1) / kThreads), grid_rows(rows));
  const size_t esz = in_f32 ? 4 : 2;
  const bool vec = ((uintptr_t)x % (4 * esz) == 0) && (ld % 4 == 0);
#define RESQ_QR(F, I, V) hipLaunchKernelGGL((quant_rows_kernel<F, I, V>), grid, dim3(kThreads), 0, s, x, rows, cols, ld, codes, scales)
  if (fmt == kMX) {
    if (in_f32) { if (vec) RESQ_QR(kMX, true, true); else RESQ_QR(kMX, true, false); }
    else { if (vec) RESQ_QR(kMX, false, true); else RESQ_QR(kMX, false, false); }
  } else {
    if (in_f32) { if (vec) RESQ_QR(kHI, true, true); else RESQ_QR(kHI, true, false); }
    else { if (vec) RESQ_QR(kHI, false, true); else RESQ_QR(kHI, false, false); }
  }
#undef RESQ_QR
}

void launch_quant_cols(int fmt, const void* x, bool in_f32, int64_t rows, int64_t cols,
                       int64_t ld, uint8_t* codes, void* scales, hipStream_t s) {
  if (rows == 0 || cols == 0) return;
  const dim3 grid((unsigned)((cols + 63) / 64), (unsigned)((rows + 63) / 64));
#define RESQ_QC(F, I) hipLaunchKernelGGL((quant_cols_kernel<F, I>), grid, dim3(kThreads), 0, s, x, rows, cols, ld, codes, scales)
  if (fmt == kMX) { if (in_f32) RESQ_QC(kMX, true); else RESQ_QC(kMX, false); }
  else { if (in_f32) RESQ_QC(kHI, true); else RESQ_QC(kHI, false); }
#undef RESQ_QC
}

void launch_residual(int fmt, int mode, const uint16_t* X, int64_t m, int64_t d, int64_t ldx,
                     uint8_t* qx_codes, void* qx_scales, uint8_t* qr_codes, void* qr_scales,
                     uint8_t* keep_mask, double* partials, hipStream_t s, bool frag) {
  if (m == 0 || d == 0) return;
  const int64_t m_rows = frag ? (m + 31) / 32 * 32 : m;
  const dim3 grid((unsigned)((d / 4 + kThreads - 1) / kThreads), grid_rows(m_rows));
  const bool vec = ((uintptr_t)X % 8 == 0) && (ldx % 4 == 0);
#define RESQ_RK(F, M, V, G) hipLaunchKernelGGL((residual_kernel<F, M, V, G>), grid, dim3(kThreads), 0, s, X, m, m_rows, d, ldx, qx_codes, qx_scales, qr_codes, qr_scales, keep_mask, partials)
#define RESQ_RK_MODE(F, V, G)                                       \
  switch (mode) {                                                   \
    case kResidNone: RESQ_RK(F, kResidNone, V, G); break;           \
    case kResidIdentity: RESQ_RK(F, kResidIdentity, V, G); break;   \
    case kResid24: RESQ_RK(F, kResid24, V, G); break;               \
    default: RESQ_RK(F, kResidDense, V, false); break;              \
  }
#define RESQ_RK_VEC(F, G) if (vec) { RESQ_RK_MODE(F, true, G) } else { RESQ_RK_MODE(F, false, G) }
  if (fmt == kMX) { if (frag) { RESQ_RK_VEC(kMX, true) } else { RESQ_RK_VEC(kMX, false) } }
  else { if (frag) { RESQ_RK_VEC(kHI, true) } else { RESQ_RK_VEC(kHI, false) } }
#undef RESQ_RK_VEC
#undef RESQ_RK_MODE
#undef RESQ_RK
}

}  // namespace resq
