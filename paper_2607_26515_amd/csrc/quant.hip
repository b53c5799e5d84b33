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
// Residual pass of Eq. 2 / Eq. 4: Q(X), dX = X - Q(X) (float32, exact), Q(dX), S_2:4
// ---------------------------------------------------------------------------------------
template <int FMT, int MODE, bool VEC>
__global__ __launch_bounds__(kThreads) void residual_kernel(
    const uint16_t* __restrict__ X, int64_t m, int64_t d, int64_t ldx,
    uint8_t* __restrict__ qx_codes, void* __restrict__ qx_scales, uint8_t* __restrict__ qr_codes,
    void* __restrict__ qr_scales, uint8_t* __restrict__ keep_mask, double* __restrict__ partials) {
  const int64_t j4 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (4 * j4 >= d) return;
  for (int64_t row = blockIdx.y; row < m; row += gridDim.y) {
    float v[4];
    load4<false, VEC>(X, row * ldx + 4 * j4, v);
    const Quad qx = quantize_quad<FMT>(v);
    *reinterpret_cast<uint16_t*>(qx_codes + row * (d / 2) + 2 * j4) = (uint16_t)pack_quad_codes(qx.code);
    store_scale<FMT>(qx_scales, row, d, j4, qx.scale);
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
      *reinterpret_cast<uint16_t*>(qr_codes + row * (d / 2) + 2 * j4) = (uint16_t)pack_quad_codes(c);
      store_scale<FMT>(qr_scales, row, d, j4, qr.scale);
      if (keep_mask != nullptr && MODE != kResidDense) {
        const uint32_t other = __shfl_xor(keep, 1, 64);
        if ((threadIdx.x & 1) == 0) keep_mask[row * (d / 8) + j4 / 2] = (uint8_t)(keep | (other << 4));
      }
      if (partials != nullptr) {
        // exact per-scale-block sum of squares (shared power-of-two factor, small integers)
        double s = 0.0;
#pragma unroll
        for (int k = 0; k < 4; ++k) s += (double)qr.val[k] * (double)qr.val[k];
        constexpr int G = (FMT == kMX) ? 8 : 16;
        s = group_sum<G>(s);
        if ((threadIdx.x & (G - 1)) == 0) partials[row * (d / (4 * G)) + j4 / G] = s;
      }
    }
  }
}

// ---------------------------------------------------------------------------------------
// HiF4 -> split E2M3 MFMA fragments.  Fragment (t, kb, term) holds, for lane l (row
// 32t + l%32, K half l/32 of 64-block kb), 32 six-bit codes in 24 bytes; term 0 = hi, 1 = lo.
// One thread per (row tile, k-block, lane).
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void pack_hif4_kernel(
    const uint8_t* __restrict__ codes, const uint32_t* __restrict__ meta, int64_t rows,
    int64_t rows_pad, int64_t K, uint8_t* __restrict__ frag, uint8_t* __restrict__ frag_c1) {
  const int64_t nkb = K / 64;
  const int64_t gid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t total = (rows_pad / 32) * nkb * 64;
  if (gid >= total) return;
  const int l = (int)(gid & 63);
  const int64_t tk = gid >> 6;  // t * nkb + kb
  const int64_t t = tk / nkb, kb = tk % nkb;
  const int64_t row = t * 32 + (l & 31);
  const int half = l >> 5;
  uint32_t hi[6] = {0, 0, 0, 0, 0, 0}, lo[6] = {0, 0, 0, 0, 0, 0};
  uint32_t c1 = 0;
  if (row < rows) {
    const uint32_t mt = meta[row * nkb + kb];
    c1 = mt & 0xFFu;
    const uint4 cw = *reinterpret_cast<const uint4*>(codes + row * (K / 2) + kb * 32 + half * 16);
    const uint32_t words[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const uint32_t code = (words[i >> 3] >> (4 * (i & 7))) & 15u;
      const int h = half * 8 + (i >> 2);  // level-3 group within the 64-block
      const int b = (int)((mt >> (8 + (h >> 1))) & 1u) + (int)((mt >> (16 + h)) & 1u);
      uint32_t ch, cl;
      hif4_split_e2m3(code, (int)c1, b, ch, cl);
      const int bit = 6 * i;
      hi[bit >> 5] |= ch << (bit & 31);
      lo[bit >> 5] |= cl << (bit & 31);
      if ((bit & 31) > 26) {  // field straddles two words
        hi[(bit >> 5) + 1] |= ch >> (32 - (bit & 31));
        lo[(bit >> 5) + 1] |= cl >> (32 - (bit & 31));
      }
    }
  }
  uint32_t* ph = reinterpret_cast<uint32_t*>(frag + ((tk * 2 + 0) * 64 + l) * 24);
  uint32_t* pl = reinterpret_cast<uint32_t*>(frag + ((tk * 2 + 1) * 64 + l) * 24);
#pragma unroll
  for (int w = 0; w < 6; ++w) { ph[w] = hi[w]; pl[w] = lo[w]; }
  frag_c1[tk * 64 + l] = (uint8_t)c1;
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
                     uint8_t* keep_mask, double* partials, hipStream_t s) {
  if (m == 0 || d == 0) return;
  const dim3 grid((unsigned)((d / 4 + kThreads - 1) / kThreads), grid_rows(m));
  const bool vec = ((uintptr_t)X % 8 == 0) && (ldx % 4 == 0);
#define RESQ_RK(F, M, V) hipLaunchKernelGGL((residual_kernel<F, M, V>), grid, dim3(kThreads), 0, s, X, m, d, ldx, qx_codes, qx_scales, qr_codes, qr_scales, keep_mask, partials)
#define RESQ_RK_MODE(F, V)                                  \
  switch (mode) {                                          \
    case kResidNone: RESQ_RK(F, kResidNone, V); break;     \
    case kResidIdentity: RESQ_RK(F, kResidIdentity, V); break; \
    case kResid24: RESQ_RK(F, kResid24, V); break;         \
    default: RESQ_RK(F, kResidDense, V); break;            \
  }
  if (fmt == kMX) { if (vec) { RESQ_RK_MODE(kMX, true) } else { RESQ_RK_MODE(kMX, false) } }
  else { if (vec) { RESQ_RK_MODE(kHI, true) } else { RESQ_RK_MODE(kHI, false) } }
#undef RESQ_RK_MODE
#undef RESQ_RK
}

void launch_pack_hif4(const uint8_t* codes, const uint32_t* meta, int64_t rows,
                      int64_t rows_pad, int64_t K, uint8_t* frag, uint8_t* frag_c1,
                      hipStream_t s) {
  const int64_t total = (rows_pad / 32) * (K / 64) * 64;
  if (total == 0) return;
  hipLaunchKernelGGL(pack_hif4_kernel, dim3((unsigned)((total + kThreads - 1) / kThreads)),
                     dim3(kThreads), 0, s, codes, meta, rows, rows_pad, K, frag, frag_c1);
}

}  // namespace resq
