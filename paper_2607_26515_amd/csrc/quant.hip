// Quantization passes: Q along rows or columns, the fused residual pass of the ResQ linear
// (Q(X), dX = X - Q(X), Q(dX), S_2:4) and the HiF4 MFMA operand packing.
#include "kernels.h"
#include "profiler.h"
#include "quant_core.h"
#include "hist.h"

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
// Residual pass of Eq. 2 / Eq. 4 with K-major output: Q(X), dX = X - Q(X) (float32,
// exact), Q(dX), and S_k:4 / S_k:8 / identity / the dense Q(dX) a global selection prunes
// later.  A lane holds 4 consecutive elements; an S_k:8 group is the lane pair (2i, 2i+1),
// which d % 8 == 0 keeps active or inactive together.
// ---------------------------------------------------------------------------------------
template <int FMT, int MODE, bool VEC>
__global__ __launch_bounds__(kThreads) void residual_kernel(
    const uint16_t* __restrict__ X, int64_t m, int64_t m_rows, int64_t d, int64_t ldx,
    uint8_t* __restrict__ qx_codes, void* __restrict__ qx_scales, uint8_t* __restrict__ qr_codes,
    void* __restrict__ qr_scales, uint8_t* __restrict__ keep_mask, double* __restrict__ partials,
    int nm_keep) {
  const int64_t j4 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (4 * j4 >= d) return;
  for (int64_t row = blockIdx.y; row < m_rows; row += gridDim.y) {
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (row < m) load4<false, VEC>(X, row * ldx + 4 * j4, v);
    const Quad qx = quantize_quad<FMT>(v);
    *reinterpret_cast<uint16_t*>(qx_codes + row * (d / 2) + 2 * j4) = (uint16_t)pack_quad_codes(qx.code);
    store_scale<FMT>(qx_scales, row, d, j4, qx.scale);
    if constexpr (MODE != kResidNone) {
      float r[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) r[k] = v[k] - qx.val[k];  // exact in float32
      const Quad qr = quantize_quad<FMT>(r);
      uint32_t keep = 0xFu;
      if constexpr (MODE == kResid24) {
        keep = keep_2_of_4(qr.code);
      } else if constexpr (MODE == kResidNM4) {
        uint32_t mag[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) mag[k] = qr.code[k] & 7u;
        keep = keep_k_of_g<4>(mag, nm_keep);
      } else if constexpr (MODE == kResidNM8) {
        // the pair's 8 codes and their shifts (HiF4 level-3 groups may differ)
        const uint32_t mine = pack_quad_codes(qr.code) | ((uint32_t)qr.b << 16);
        const uint32_t other = __shfl_xor(mine, 1, 64);
        const bool odd = (threadIdx.x & 1) != 0;
        const uint32_t lo = odd ? other : mine, hi = odd ? mine : other;
        uint32_t c8[8];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          c8[k] = (lo >> (4 * k)) & 15u;
          c8[4 + k] = (hi >> (4 * k)) & 15u;
        }
        const int b2[2] = {(int)(lo >> 16), (int)(hi >> 16)};
        keep = (keep_local8<8>(c8, b2, nm_keep) >> (odd ? 4 : 0)) & 0xFu;
      }
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

// ---------------------------------------------------------------------------------------
// Residual pass writing MFMA fragments: one workgroup of 256 threads per fragment (row tile
// t, K step kb).  Fragment lane record r (row 32t + r%32, elements 64kb + 32(r/32) .. +31)
// is handled by 4 threads of 8 elements each; thread i of the workgroup takes row i/8 of the
// tile, half (i/4)%2 and the 8-element slice i%4.  An MXFP4 scale block (32 elements) is 4
// consecutive lanes, a HiF4 64-block 8 consecutive lanes, a HiF4 level-2 group one lane.
// Each thread quantizes its slice, forms dX = X - Q(X) (exact in float32), quantizes dX,
// applies S_k:4 or S_k:8 (whole groups inside the slice), and the 4 threads of a record write it as one contiguous 16-byte (MXFP4) or
// 48-byte (HiF4 E2M3 hi | lo) run.  Rows past m, and the missing half of an MXFP4 K step
// when d % 64 == 32, quantize zeros.
// ---------------------------------------------------------------------------------------
template <int FMT>
__device__ __forceinline__ void quantize8(const float x[8], uint32_t code[8], float val[8],
                                          uint32_t& scale_byte, int& c1, int b[2], int& b2o) {
  float a = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) a = fmaxf(a, fabsf(x[i]));
  if constexpr (FMT == kMX) {
    const int E = mx_exponent(group_max<4>(a));
    scale_byte = (uint32_t)(E + 127);
    c1 = 0;
    b[0] = b[1] = 0;
    b2o = 0;
    const float sc = mx_scale_f32(E);
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
      const uint32_t c2 = mx_code2(x[i], x[i + 1], sc);
      code[i] = c2 & 15u;
      code[i + 1] = c2 >> 4;
      mx_value2(c2, sc, val[i], val[i + 1]);
    }
  } else {
    c1 = hif4_c1(group_max<8>(a));
    scale_byte = (uint32_t)c1;
    const float fit0 = hif4_half_fit(c1, 0), fit1 = hif4_half_fit(c1, 1);
    const int b2 = a <= fit0 ? 1 : 0;  // this lane's 8 elements are one level-2 group
    b2o = b2;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      float a4 = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) a4 = fmaxf(a4, fabsf(x[4 * hh + e]));
      b[hh] = b2 + (a4 <= (b2 ? fit1 : fit0) ? 1 : 0);
    }
    const Hif4Mid mid = hif4_mid(c1);
    const float step[2] = {hif4_step(c1, b[0]), hif4_step(c1, b[1])};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t k = hif4_k(x[i], c1, b[i / 4], mid);
      code[i] = ((__float_as_uint(x[i]) >> 28) & 8u) | k;
      val[i] = hif4_signed_value(k, step[i / 4], x[i]);
    }
  }
}

// The 4 threads of lane record `rec` (slice s = lane % 4) write it.
template <int FMT>
__device__ __forceinline__ void store_record8(uint8_t* __restrict__ frag, uint8_t* __restrict__ fsc,
                                              int64_t rec, int s, const uint32_t code[8],
                                              uint32_t scale_byte, int c1, const int b[2]) {
  if constexpr (FMT == kMX) {
    uint32_t w = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) w |= code[i] << (4 * i);
    reinterpret_cast<uint32_t*>(frag + rec * 16)[s] = w;
  } else {
    // 8 six-bit fields = 48 bits each of hi and lo; record = hi bits [0,192) then lo.  Each
    // 48-bit run is built as two 24-bit runs of 4 fields (one level-3 shift each) in 32-bit
    // words.
    uint32_t rh[2], rl[2];
    const uint32_t q2 = (4u + ((uint32_t)c1 & 3u)) * 0x00010001u;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const uint32_t nb = code[4 * hh] | (code[4 * hh + 1] << 8) | (code[4 * hh + 2] << 16) | (code[4 * hh + 3] << 24);
      hif4_split4(nb, q2, (uint32_t)b[hh], rh[hh], rl[hh]);
    }
    const uint64_t h = rh[0] | ((uint64_t)rh[1] << 24), l = rl[0] | ((uint64_t)rl[1] << 24);
    // thread s writes record dwords 3s .. 3s+2: hi of slices 0,1 / hi of 2,3 / lo of 0,1 /
    // lo of 2,3, i.e. 96 bits assembled from two slices' 48-bit runs
    const int lane = __lane_id();
    const int base = lane & ~3, src = base + 2 * (s & 1);
    const uint32_t hl0 = __shfl((uint32_t)h, src, 64), hh0 = __shfl((uint32_t)(h >> 32), src, 64);
    const uint32_t hl1 = __shfl((uint32_t)h, src + 1, 64), hh1 = __shfl((uint32_t)(h >> 32), src + 1, 64);
    const uint32_t ll0 = __shfl((uint32_t)l, src, 64), lh0 = __shfl((uint32_t)(l >> 32), src, 64);
    const uint32_t ll1 = __shfl((uint32_t)l, src + 1, 64), lh1 = __shfl((uint32_t)(l >> 32), src + 1, 64);
    const bool lo_part = s >= 2;
    const uint64_t p0 = ((uint64_t)(lo_part ? lh0 : hh0) << 32) | (lo_part ? ll0 : hl0);  // 48 bits
    const uint64_t p1 = ((uint64_t)(lo_part ? lh1 : hh1) << 32) | (lo_part ? ll1 : hl1);
    const uint32_t d0 = (uint32_t)p0;
    const uint32_t d1 = (uint32_t)(p0 >> 32) | ((uint32_t)p1 << 16);
    const uint32_t d2 = (uint32_t)(p1 >> 16);
    uint32_t* w = reinterpret_cast<uint32_t*>(frag + rec * 48) + 3 * s;
    w[0] = d0;
    w[1] = d1;
    w[2] = d2;
  }
  if (s == 0) fsc[rec] = (uint8_t)scale_byte;
}

// K-major output of one thread's 8 codes (row `row`, elements 64kb + 32half + 8s .. +7) for
// a global selection: the codes as one 32-bit word, the block's scale (MXFP4: the E8M0 byte
// of the 32-element half; HiF4: the metadata word of the 64-block, assembled from the 8
// lanes of the row, lane g = level-2 group g), and the exact per-scale-block sum of squares
// of the dequantized values.  Every lane must call this (ballots, shuffles); `in` = the
// elements lie inside the matrix.
__device__ __forceinline__ uint32_t spread8(uint32_t x) {  // bit i -> bit 2i
  x = (x | (x << 4)) & 0x0F0Fu;
  x = (x | (x << 2)) & 0x3333u;
  return (x | (x << 1)) & 0x5555u;
}

template <int FMT>
__device__ __forceinline__ void store_kmajor8(uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                              double* __restrict__ partials, bool in, int64_t row,
                                              int64_t d, int64_t kb, int half, int s,
                                              const uint32_t code[8], const float val[8],
                                              uint32_t scale_byte, const int b[2], int b2,
                                              double* __restrict__ rowsq = nullptr) {
  const int64_t col0 = kb * 64 + 32 * half + 8 * s;
  uint32_t w = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) w |= code[i] << (4 * i);
  if (in) *reinterpret_cast<uint32_t*>(codes + row * (d / 2) + col0 / 2) = w;
  double sq = 0.0;  // exact: squares of a shared scale times small integers
#pragma unroll
  for (int i = 0; i < 8; ++i) sq += (double)val[i] * (double)val[i];
  if constexpr (FMT == kMX) {
    sq = group_sum<4>(sq);
    if (in && s == 0) {
      scales[row * (d / 32) + kb * 2 + half] = (uint8_t)scale_byte;
      if (partials) partials[row * (d / 32) + kb * 2 + half] = sq;
    }
    if (rowsq && s == 0) rowsq[half] = in ? sq : 0.0;  // this row's sum of scale block `half`
  } else {
    const int base = __lane_id() & ~7;  // the row's 8 lanes
    const uint32_t bits2 = (uint32_t)(__ballot(b2 != 0) >> base) & 0xFFu;
    const uint32_t b3a = (uint32_t)(__ballot(b[0] != b2) >> base) & 0xFFu;
    const uint32_t b3b = (uint32_t)(__ballot(b[1] != b2) >> base) & 0xFFu;
    const uint32_t meta = scale_byte | (bits2 << 8) | ((spread8(b3a) | (spread8(b3b) << 1)) << 16);
    sq = group_sum<8>(sq);
    if (in && half == 0 && s == 0) {
      reinterpret_cast<uint32_t*>(scales)[row * (d / 64) + kb] = meta;
      if (partials) partials[row * (d / 64) + kb] = sq;
    }
    if (rowsq && half == 0 && s == 0) rowsq[0] = in ? sq : 0.0;  // this row's sum of the 64-block
  }
}

// The bf16 nearest to a float64 (ties to even), in one rounding: round to float32 with
// round-to-odd (the float32 grid has 16 more bits than bf16's, so the sticky lowest bit keeps
// every tie decision of the final step), then round that to bf16 to nearest even.  Values past
// the largest finite bf16 give inf.
__device__ __forceinline__ float f64_to_bf16_value(double v) {
  float f = (float)v;
  if ((double)f != v) {
    uint32_t b = __float_as_uint(f);
    if (fabs((double)f) > fabs(v)) b -= 1u;  // rounded away from zero: step back
    f = __uint_as_float(b | 1u);
  }
  const uint32_t u = __float_as_uint(f);
  return __uint_as_float(((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16) << 16);
}

// X = silu(G) * U for 8 consecutive elements: float64 sigmoid and product, one rounding.
template <bool VEC>
__device__ __forceinline__ void swiglu8(const Producer& p, int64_t row, int64_t col0, float x[8]) {
  float g[8], u[8];
  if (p.f32) {
    const float* gs = reinterpret_cast<const float*>(p.g) + row * p.ldg + col0;
    const float* us = reinterpret_cast<const float*>(p.u) + row * p.ldu + col0;
    if constexpr (VEC) {
      const float4 g0 = reinterpret_cast<const float4*>(gs)[0], g1 = reinterpret_cast<const float4*>(gs)[1];
      const float4 u0 = reinterpret_cast<const float4*>(us)[0], u1 = reinterpret_cast<const float4*>(us)[1];
      g[0] = g0.x; g[1] = g0.y; g[2] = g0.z; g[3] = g0.w; g[4] = g1.x; g[5] = g1.y; g[6] = g1.z; g[7] = g1.w;
      u[0] = u0.x; u[1] = u0.y; u[2] = u0.z; u[3] = u0.w; u[4] = u1.x; u[5] = u1.y; u[6] = u1.z; u[7] = u1.w;
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) { g[i] = gs[i]; u[i] = us[i]; }
    }
  } else {
    const uint16_t* gs = reinterpret_cast<const uint16_t*>(p.g) + row * p.ldg + col0;
    const uint16_t* us = reinterpret_cast<const uint16_t*>(p.u) + row * p.ldu + col0;
    if constexpr (VEC) {
      const uint4 gw = *reinterpret_cast<const uint4*>(gs), uw = *reinterpret_cast<const uint4*>(us);
      const uint32_t gv[4] = {gw.x, gw.y, gw.z, gw.w}, uv[4] = {uw.x, uw.y, uw.z, uw.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        g[2 * e] = bf16_to_f32(gv[e] & 0xFFFFu); g[2 * e + 1] = bf16_to_f32(gv[e] >> 16);
        u[2 * e] = bf16_to_f32(uv[e] & 0xFFFFu); u[2 * e + 1] = bf16_to_f32(uv[e] >> 16);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) { g[i] = bf16_to_f32(gs[i]); u[i] = bf16_to_f32(us[i]); }
    }
  }
  // Fast path in float32: e = expf(-g) (about 1 ulp), 1 + e, g / (1 + e) and the product
  // with u (0.5 ulp each) put s within 5 float32 ulps of the exact value (e's error enters
  // silu scaled by e / (1 + e) <= 1).  A bf16 midpoint lies 2^15 float32 ulps from each bf16
  // value, so when s is more than 64 ulps from the nearest midpoint its bf16 rounding is that
  // of the exact value.  The rest (about 0.2% of elements), and inputs outside the bound's
  // premises (g < -80, where exp(-g) nears float32 overflow; 0 < |g| < 2^-100, where g / 2
  // may lose bits; a non-finite s), take the float64 path one element at a time, so a wave
  // repeats it only as often as its busiest lane needs it.
  uint32_t pending = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float gi = g[i];
    const float sv = gi / (1.0f + expf(-gi)) * u[i];
    const uint32_t b = __float_as_uint(sv);
    const int dist = abs((int)(b & 0xFFFFu) - 0x8000);
    const bool premise = gi >= -80.f && (gi == 0.f || fabsf(gi) >= 0x1p-100f) && isfinite(sv);
    if (premise && dist > 64) {
      x[i] = __uint_as_float(((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16) << 16);
    } else {
      pending |= 1u << i;
    }
  }
  while (pending != 0) {
    const int i = __builtin_ctz(pending);
    pending &= pending - 1u;
    float gi = 0.f, ui = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (k == i) { gi = g[k]; ui = u[k]; }
    const double gd = (double)gi;
    const float xv = f64_to_bf16_value(gd / (1.0 + exp(-gd)) * (double)ui);
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (k == i) x[k] = xv;
  }
}

// ---------------------------------------------------------------------------------------
// RMSNorm producer.  Float32 steps rounded to nearest even, each checked exactly: a float64
// result rounded to float32 is within one place of the right answer, and the exact comparison
// with the midpoints next to it (products of at most 25 x 25 bits, exact in float64) fixes
// the last place.  Neither a quotient of float32 values nor a square root of one can fall on
// a midpoint, so there are no ties.
// ---------------------------------------------------------------------------------------
__device__ __forceinline__ float f32_up(float x) { return __uint_as_float(__float_as_uint(x) + 1u); }
__device__ __forceinline__ float f32_down(float x) { return __uint_as_float(__float_as_uint(x) - 1u); }

// a / b to nearest, for a >= 0 and b > 0 (inf allowed in one of them)
__device__ float div_rn_f32(float a, float b) {
  float z = (float)((double)a / (double)b);
  if (!isfinite(z) || !isfinite(b)) return z;
  if (0.5 * ((double)z + (double)f32_up(z)) * (double)b < (double)a) return f32_up(z);
  if (z > 0.f && 0.5 * ((double)z + (double)f32_down(z)) * (double)b > (double)a) return f32_down(z);
  return z;
}

// sqrt(t) to nearest, for t >= 0 (inf allowed)
__device__ float sqrt_rn_f32(float t) {
  float z = (float)sqrt((double)t);
  if (!isfinite(z)) return z;
  const double hi = 0.5 * ((double)z + (double)f32_up(z));
  if (hi * hi < (double)t) return f32_up(z);
  const double lo = 0.5 * ((double)z + (double)f32_down(z));
  if (z > 0.f && lo * lo > (double)t) return f32_down(z);
  return z;
}

// A bf16 value is M * 2^(E - 134) with M < 2^8 (E = the exponent field, 1 for subnormals), so
// its square is M^2 * 2^(2E - 268).  One row's squares are added as integers per exponent
// field (LDS histograms in kLdsCopies per-lane copies, hist.h; a copy's bin gets at most
// d / 8 squares below 2^16, under 2^32 for d <= 2^18), the 255 bin totals are added into an
// integer of kRmsLimbs 32-bit limbs in
// units of 2^-268 (bin E at bit 2E, below 2^(2 * 255 + 34) < 2^(32 * kRmsLimbs)), and that
// exact sum is rounded once: to 53 bits by truncation with the sticky lowest bit (round to
// odd), then to float32 to nearest even, which gives the float32 nearest to the exact sum
// (53 >= 24 + 2 bits).
constexpr int kRmsLimbs = 18;

__device__ float rms_row_factor(const unsigned long long* limb, int64_t d, float eps) {
  uint32_t n[kRmsLimbs];
  unsigned long long carry = 0;
#pragma unroll
  for (int l = 0; l < kRmsLimbs; ++l) {
    const unsigned long long v = limb[l] + carry;
    n[l] = (uint32_t)v;
    carry = v >> 32;
  }
  int top = kRmsLimbs - 1;
  while (top >= 0 && n[top] == 0u) --top;
  float s = 0.f;
  if (top >= 0) {
    const int lz = __clz(n[top]);
    const int msb = 32 * top + 31 - lz;  // the sum lies in [2^(msb - 268), 2^(msb - 267))
    const uint32_t x1 = top >= 1 ? n[top - 1] : 0u, x0 = top >= 2 ? n[top - 2] : 0u;
    unsigned long long w = ((((unsigned long long)n[top]) << 32) | x1) << lz;  // msb at bit 63
    bool sticky;
    if (lz > 0) {
      w |= x0 >> (32 - lz);
      sticky = (x0 << lz) != 0u;
    } else {
      sticky = x0 != 0u;
    }
    for (int l = 0; l < top - 2; ++l) sticky |= n[l] != 0u;
    unsigned long long sig = w >> 11;
    sticky |= (w & 0x7FFull) != 0ull;
    if (sticky) sig |= 1ull;
    s = (float)ldexp((double)sig, msb - 52 - 268);  // exact in float64, then one rounding
  }
  const float mu = div_rn_f32(s, (float)d);
  const float t = mu + eps;
  return div_rn_f32(1.f, sqrt_rn_f32(t));
}

// grid-stride over rows, one workgroup of 256 threads per row at a time
template <bool VEC>
__global__ __launch_bounds__(256) void rms_rows_kernel(const uint16_t* __restrict__ H, int64_t m,
                                                        int64_t d, int64_t ldh, float eps,
                                                        float* __restrict__ rinv) {
  __shared__ uint32_t wh[kLdsCopies * 257];
  __shared__ unsigned long long limb[kRmsLimbs];
  const int tid = threadIdx.x;
  uint32_t* hc = wh + (tid % kLdsCopies) * 257;  // this lane's copy
  for (int64_t row = blockIdx.x; row < m; row += gridDim.x) {
    for (int i = tid; i < kLdsCopies * 257; i += 256) wh[i] = 0u;
    if (tid < kRmsLimbs) limb[tid] = 0ull;
    __syncthreads();
    const uint16_t* src = H + row * ldh;
    for (int64_t c = (int64_t)tid * 8; c < d; c += 256 * 8) {  // d % 8 == 0
      uint32_t b[8];
      if constexpr (VEC) {
        const uint4 u = *reinterpret_cast<const uint4*>(src + c);
        const uint32_t v[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) { b[2 * e] = v[e] & 0xFFFFu; b[2 * e + 1] = v[e] >> 16; }
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) b[i] = src[c + i];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t e = (b[i] >> 7) & 0xFFu;
        const uint32_t mant = (b[i] & 0x7Fu) | (e ? 0x80u : 0u);
        if (mant) atomicAdd(&hc[e ? e : 1u], mant * mant);
      }
    }
    __syncthreads();
    // bin tid (0 .. 255) at bit 2 * tid: three 32-bit pieces into three limbs
    unsigned long long T = 0;  // up to 2^18 squares below 2^16: 64-bit
#pragma unroll
    for (int c = 0; c < kLdsCopies; ++c) T += wh[c * 257 + tid];
    if (T) {
      const int off = 2 * tid, L = off >> 5, sh = off & 31;
      const unsigned long long lo = (T & 0xFFFFFFFFull) << sh, hi = (T >> 32) << sh;
      atomicAdd(&limb[L], lo & 0xFFFFFFFFull);
      atomicAdd(&limb[L + 1], (lo >> 32) + (hi & 0xFFFFFFFFull));
      if (hi >> 32) atomicAdd(&limb[L + 2], hi >> 32);
    }
    __syncthreads();
    if (tid == 0) rinv[row] = rms_row_factor(limb, d, eps);
    __syncthreads();  // the next row clears the histograms and limbs
  }
}

// X = RMSNorm(H) * gamma for 8 consecutive elements of one row
template <bool VEC>
__device__ __forceinline__ void rmsnorm8(const Producer& p, int64_t row, int64_t col0, float x[8]) {
  const uint16_t* hs = reinterpret_cast<const uint16_t*>(p.g) + row * p.ldg + col0;
  const uint16_t* gs = reinterpret_cast<const uint16_t*>(p.u) + col0;
  const float r = p.rinv[row];
  float h[8], g[8];
  if constexpr (VEC) {
    const uint4 hw = *reinterpret_cast<const uint4*>(hs), gw = *reinterpret_cast<const uint4*>(gs);
    const uint32_t hv[4] = {hw.x, hw.y, hw.z, hw.w}, gv[4] = {gw.x, gw.y, gw.z, gw.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      h[2 * e] = bf16_to_f32(hv[e] & 0xFFFFu); h[2 * e + 1] = bf16_to_f32(hv[e] >> 16);
      g[2 * e] = bf16_to_f32(gv[e] & 0xFFFFu); g[2 * e + 1] = bf16_to_f32(gv[e] >> 16);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) { h[i] = bf16_to_f32(hs[i]); g[i] = bf16_to_f32(gs[i]); }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float y = h[i] * r;   // two separate float32 products, each rounded
    const uint32_t u = __float_as_uint(y * g[i]);
    x[i] = __uint_as_float(((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16) << 16);
  }
}

// Row tile t, K step kb of the fused residual pass (one workgroup of 256 threads).  PROD
// (a ProducerKind, or 0): X comes from the producer `prod` instead of from X.
template <int FMT, int MODE, bool VEC, int PROD>
__device__ __forceinline__ void residual_frag_tile(
    const uint16_t* __restrict__ X, int64_t m, int64_t d, int64_t ldx, int64_t nkb,
    uint8_t* __restrict__ fx, uint8_t* __restrict__ fsx, uint8_t* __restrict__ fr,
    uint8_t* __restrict__ fsr, double* __restrict__ partials, int nm_keep, const Producer& prod,
    int64_t t, int64_t kb, uint32_t* ehist_lds, double* rowsq_lds, double* __restrict__ bkeys) {
  const int64_t f = t * nkb + kb;  // fragment index
  const int tid = threadIdx.x;
  const int rr = tid >> 3, half = (tid >> 2) & 1, s = tid & 3;
  const int64_t row = t * 32 + rr;
  const int64_t col0 = kb * 64 + 32 * half + 8 * s;
  float x[8];
  if (PROD == kProdSwiglu && row < m && col0 < d) {
    swiglu8<VEC>(prod, row, col0, x);
  } else if (PROD == kProdRmsnorm && row < m && col0 < d) {
    rmsnorm8<VEC>(prod, row, col0, x);
  } else if (row < m && col0 < d) {
    const uint16_t* src = X + row * ldx + col0;
    if constexpr (VEC) {
      const uint4 u = *reinterpret_cast<const uint4*>(src);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[2 * e] = bf16_to_f32(w[e] & 0xFFFFu);
        x[2 * e + 1] = bf16_to_f32(w[e] >> 16);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = bf16_to_f32(src[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = 0.f;
  }
  const int64_t rec = f * 64 + rr + 32 * half;
  uint32_t code[8], scale_byte;
  float val[8];
  int c1, b[2], b2;
  quantize8<FMT>(x, code, val, scale_byte, c1, b, b2);
  store_record8<FMT>(fx, fsx, rec, s, code, scale_byte, c1, b);
  if constexpr (MODE != kResidNone) {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] -= val[i];  // dX, exact in float32
    quantize8<FMT>(x, code, val, scale_byte, c1, b, b2);
    if constexpr (MODE == kResid24) {
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const uint32_t c4[4] = {code[4 * g], code[4 * g + 1], code[4 * g + 2], code[4 * g + 3]};
        const uint32_t keep = keep_2_of_4(c4);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (!((keep >> e) & 1u)) code[4 * g + e] = 0u;
      }
    } else if constexpr (MODE == kResidNM4 || MODE == kResidNM8) {
      const uint32_t keep = keep_local8<MODE == kResidNM4 ? 4 : 8>(code, b, nm_keep);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (!((keep >> e) & 1u)) code[e] = 0u;
    }
    if constexpr (MODE == kResidDense) {
      store_kmajor8<FMT>(fr, fsr, partials, row < m && col0 < d, row, d, kb, half, s, code, val,
                         scale_byte, b, b2, bkeys ? rowsq_lds + 2 * rr : nullptr);
      if (bkeys) {  // workgroup-uniform
        // the key of 32 x 64 block (t, kb): its rows' scale-block sums, rows in order, scale
        // blocks in column order (the order the selection defines)
        __syncthreads();
        if (threadIdx.x == 0) {
          double acc = 0.0;
          for (int i = 0; i < 32; ++i)
            if (t * 32 + i < m)
#pragma unroll
              for (int q = 0; q < (FMT == kMX ? 2 : 1); ++q) acc += rowsq_lds[2 * i + q];
          bkeys[t * (d / 64) + kb] = acc;
        }
        __syncthreads();  // the row sums are overwritten by the next row tile
      }
      if (ehist_lds) {  // workgroup-uniform
        // the element-wise selection's first histogram: exponent fields of |Q(dX)|, exactly
        // the keys its passes decode from these codes (one float32 per value)
#pragma unroll
        for (int i = 0; i < 8; ++i)
          hist_add_copies(ehist_lds, 256, (__float_as_uint(val[i]) >> 23) & 255u, row < m && col0 < d);
      }
    } else {
      store_record8<FMT>(fr, fsr, rec, s, code, scale_byte, c1, b);
    }
  }
}

// grid: x = K step, y = row tiles (grid-stride).  kResidDense (a global selection follows):
// fr / fsr receive the K-major Q(dX) codes and scales and `partials` its per-scale-block
// sums of squares (may be null); with ehist (element-wise selection, cleared beforehand) the
// workgroup also counts the exponent fields of |Q(dX)| and adds them into copy
// (workgroup % kElemHistCopies) of that histogram; with bkeys (block selection) it writes the
// key of each 32 x 64 block it covers (d % 64 == 0).
template <int FMT, int MODE, bool VEC, int PROD>
__global__ __launch_bounds__(256) void residual_frag_kernel(
    const uint16_t* __restrict__ X, int64_t m, int64_t d, int64_t ldx, int64_t nkb,
    uint8_t* __restrict__ fx, uint8_t* __restrict__ fsx, uint8_t* __restrict__ fr,
    uint8_t* __restrict__ fsr, double* __restrict__ partials, uint32_t* __restrict__ ehist,
    int nm_keep, Producer prod, double* __restrict__ bkeys) {
  __shared__ uint32_t lh[MODE == kResidDense ? kLdsCopies * 257 : 1];  // hist.h copies of 256 bins
  __shared__ double rowsq[MODE == kResidDense ? 64 : 1];  // block keys: the tile's row sums
  const bool counting = MODE == kResidDense && ehist != nullptr;
  if (counting) {
    for (int i = threadIdx.x; i < kLdsCopies * 257; i += 256) lh[i] = 0u;
    __syncthreads();
  }
  const int64_t mtiles = (m + 31) / 32;
  for (int64_t t = blockIdx.y; t < mtiles; t += gridDim.y)
    residual_frag_tile<FMT, MODE, VEC, PROD>(X, m, d, ldx, nkb, fx, fsx, fr, fsr, partials, nm_keep,
                                               prod, t, blockIdx.x, counting ? lh : nullptr, rowsq,
                                               MODE == kResidDense ? bkeys : nullptr);
  if (counting) {
    __syncthreads();
    const uint32_t c = hist_sum_copies(lh, 256, threadIdx.x);
    const uint32_t wg = blockIdx.y * gridDim.x + blockIdx.x;
    if (c) atomicAdd(&ehist[(wg % kElemHistCopies) * kElemHistBins + threadIdx.x], c);
  }
}

// ---------------------------------------------------------------------------------------
// Q along columns written as MFMA fragments.  The operand's rows are x's columns and its K
// axis is x's rows (blocks along the rows of x).  One workgroup per 64-row x 128-column
// tile of x, i.e. K step kb of the four operand row tiles 4T .. 4T+3: the tile is staged in
// LDS with 16-byte loads, then for each row tile every thread quantizes 8 consecutive K
// elements of one operand row with the thread -> (row, half, slice) map of
// residual_frag_kernel and writes its part of the lane record.  Rows of x past R (the
// missing half of an MXFP4 K step) and columns past C quantize zeros.
// ---------------------------------------------------------------------------------------

// HiF4 weight-side record: the 4 threads of lane record `rec` hold 8 BF6 E3M2 fields each
// (48 bits); threads s and s+1 (s even) write record dwords 3s/2 .. 3s/2+2.
__device__ __forceinline__ void store_record8_e3m2(uint8_t* __restrict__ frag, uint8_t* __restrict__ fsc,
                                                   int64_t rec, int s, const uint32_t code[8],
                                                   uint32_t scale_byte, const int b[2]) {
  uint32_t r[2];  // two 24-bit runs of 4 fields
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
    r[hh] = hif4_e3m2x4(code[4 * hh] | (code[4 * hh + 1] << 8) | (code[4 * hh + 2] << 16) | (code[4 * hh + 3] << 24),
                        (uint32_t)b[hh]);
  const uint64_t h = r[0] | ((uint64_t)r[1] << 24);
  const uint32_t plo = __shfl_xor((uint32_t)h, 1, 64), phi = __shfl_xor((uint32_t)(h >> 32), 1, 64);
  if ((s & 1) == 0) {
    const uint64_t p1 = ((uint64_t)phi << 32) | plo;  // the odd partner's 48 bits
    uint32_t* w = reinterpret_cast<uint32_t*>(frag + rec * 24) + 3 * (s >> 1);
    w[0] = (uint32_t)h;
    w[1] = (uint32_t)(h >> 32) | ((uint32_t)p1 << 16);
    w[2] = (uint32_t)(p1 >> 16);
  }
  if (s == 0) fsc[rec] = (uint8_t)scale_byte;
}

// With DUAL, the same tile also yields the row quantization (blocks along the columns of x)
// as fragments of the operand [R][C]: row tiles 2kb, 2kb+1 and K steps 2T, 2T+1 (written
// to rfrag / rfsc, activation layout), so x is read once for both.
// Operand row tiles 4T .. 4T+3, K step kb (one workgroup of 256 threads; `tile` is its
// 64 x 128 staging buffer).
template <int FMT, int PMODE, bool VEC, bool DUAL>
__device__ __forceinline__ void quant_cols_frag_tile(const uint16_t* __restrict__ x, int64_t R,
                                                     int64_t C, int64_t ld, int64_t nkb, int64_t nt,
                                                     uint8_t* __restrict__ frag, uint8_t* __restrict__ fsc,
                                                     uint8_t* __restrict__ rfrag, uint8_t* __restrict__ rfsc,
                                                     uint16_t* tile, int64_t T, int64_t kb) {
  constexpr int kPitch = 128 + 2;  // bf16 per LDS row (padding spreads the column reads)
  const int64_t r0 = kb * 64, c0 = T * 128;
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int idx = tid + 256 * q, rr = idx >> 4, cc = (idx & 15) * 8;
    const int64_t row = r0 + rr, col = c0 + cc;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    if (row < R) {
      const uint16_t* src = x + row * ld + col;
      if (VEC && col + 8 <= C) {
        const uint4 u = *reinterpret_cast<const uint4*>(src);
        w[0] = u.x; w[1] = u.y; w[2] = u.z; w[3] = u.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (col + e < C) w[e >> 1] |= (uint32_t)src[e] << (16 * (e & 1));
      }
    }
    uint32_t* dst = reinterpret_cast<uint32_t*>(tile + rr * kPitch + cc);  // 4-byte aligned
#pragma unroll
    for (int e = 0; e < 4; ++e) dst[e] = w[e];
  }
  __syncthreads();
  const int rr = tid >> 3, half = (tid >> 2) & 1, s = tid & 3;
#pragma unroll
  for (int tt = 0; tt < 4; ++tt) {
    const int64_t t = T * 4 + tt;
    if (t >= nt) break;  // uniform over the workgroup
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = bf16_to_f32(tile[(32 * half + 8 * s + e) * kPitch + 32 * tt + rr]);
    uint32_t code[8], scale_byte;
    float val[8];
    int c1, b[2], b2;
    quantize8<FMT>(v, code, val, scale_byte, c1, b, b2);
    const int64_t rec = (t * nkb + kb) * 64 + rr + 32 * half;
    if constexpr (PMODE == kPackHiB) store_record8_e3m2(frag, fsc, rec, s, code, scale_byte, b);
    else store_record8<FMT>(frag, fsc, rec, s, code, scale_byte, c1, b);
  }
  if constexpr (DUAL) {
    const int64_t rkb = (C + 63) / 64, rnt = (R + 31) / 32;  // row operand: K steps, row tiles
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int rt = q >> 1, ks = q & 1;
      const int64_t t = 2 * kb + rt, k = 2 * T + ks;
      if (t >= rnt || k >= rkb) continue;  // uniform over the workgroup
      const uint32_t* src = reinterpret_cast<const uint32_t*>(tile + (32 * rt + rr) * kPitch + 64 * ks + 32 * half + 8 * s);
      float v[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t w = src[e];
        v[2 * e] = bf16_to_f32(w & 0xFFFFu);
        v[2 * e + 1] = bf16_to_f32(w >> 16);
      }
      uint32_t code[8], scale_byte;
      float val[8];
      int c1, b[2], b2;
      quantize8<FMT>(v, code, val, scale_byte, c1, b, b2);
      store_record8<FMT>(rfrag, rfsc, (t * rkb + k) * 64 + rr + 32 * half, s, code, scale_byte, c1, b);
    }
  }
}

// grid: x = K step, y = groups of four operand row tiles (grid-stride)
template <int FMT, int PMODE, bool VEC, bool DUAL>
__global__ __launch_bounds__(256) void quant_cols_frag_kernel(const uint16_t* __restrict__ x, int64_t R,
                                                              int64_t C, int64_t ld, int64_t nkb,
                                                              int64_t nt, uint8_t* __restrict__ frag,
                                                              uint8_t* __restrict__ fsc,
                                                              uint8_t* __restrict__ rfrag,
                                                              uint8_t* __restrict__ rfsc) {
  constexpr int kPitch = 128 + 2;
  __shared__ uint16_t tile[64 * kPitch];
  const int64_t ngroups = (nt + 3) / 4;
  for (int64_t T = blockIdx.y; T < ngroups; T += gridDim.y) {
    if (T != blockIdx.y) __syncthreads();  // the previous group's reads of the tile are done
    quant_cols_frag_tile<FMT, PMODE, VEC, DUAL>(x, R, C, ld, nkb, nt, frag, fsc, rfrag, rfsc, tile, T, blockIdx.x);
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

void launch_quant_cols_frag(int mode, const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                            uint8_t* frag, uint8_t* fscale, hipStream_t s, uint8_t* rfrag,
                            uint8_t* rfscale) {
  if (rows == 0 || cols == 0) return;
  const int64_t nkb = (rows + 63) / 64, nt = (cols + 31) / 32;
  const dim3 grid((unsigned)nkb, grid_rows((nt + 3) / 4));
  const bool vec = ((uintptr_t)x % 16 == 0) && (ld % 8 == 0);
  const bool dual = rfrag != nullptr;
#define RESQ_QCF(F, P, V, D) hipLaunchKernelGGL((quant_cols_frag_kernel<F, P, V, D>), grid, dim3(256), 0, s, x, rows, cols, ld, nkb, nt, frag, fscale, rfrag, rfscale)
#define RESQ_QCF_V(F, P)                                                                   \
  if (dual) { if (vec) RESQ_QCF(F, P, true, true); else RESQ_QCF(F, P, false, true); }    \
  else { if (vec) RESQ_QCF(F, P, true, false); else RESQ_QCF(F, P, false, false); }
  if (mode == kPackMx) { RESQ_QCF_V(kMX, kPackMx) }
  else if (mode == kPackHiA) { RESQ_QCF_V(kHI, kPackHiA) }
  else { if (vec) RESQ_QCF(kHI, kPackHiB, true, false); else RESQ_QCF(kHI, kPackHiB, false, false); }
#undef RESQ_QCF_V
#undef RESQ_QCF
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

void launch_rms_rows(const uint16_t* H, int64_t m, int64_t d, int64_t ldh, float eps, float* rinv,
                     hipStream_t s) {
  if (m == 0) return;
  const unsigned grid = (unsigned)(m < 8192 ? m : 8192);
  if ((uintptr_t)H % 16 == 0 && ldh % 8 == 0)
    launch_timed(rms_rows_kernel<true>, dim3(grid), dim3(256), 0u, s, H, m, d, ldh, eps, rinv);
  else
    launch_timed(rms_rows_kernel<false>, dim3(grid), dim3(256), 0u, s, H, m, d, ldh, eps, rinv);
}

void launch_residual(int fmt, int mode, const uint16_t* X, int64_t m, int64_t d, int64_t ldx,
                     uint8_t* qx_codes, void* qx_scales, uint8_t* qr_codes, void* qr_scales,
                     uint8_t* keep_mask, double* partials, hipStream_t s, bool frag,
                     uint32_t* ehist, int nm_keep, const Producer* prod, double* bkeys) {
  if (m == 0 || d == 0) return;
  if (frag) {
    const int64_t nkb = (d + 63) / 64;
    const dim3 grid((unsigned)nkb, grid_rows((m + 31) / 32));
    const Producer pr = prod ? *prod : Producer{nullptr, nullptr, 0, 0, false, 0, nullptr};
    // 16-byte loads: 8 bf16 of X (or of G and U, or of H and gamma), or 2 x 4 floats of G and U
    const int64_t ve = prod ? (prod->f32 ? 4 : 8) : 8;
    const bool vec16 = prod ? ((uintptr_t)pr.g % 16 == 0 && (uintptr_t)pr.u % 16 == 0 &&
                               pr.ldg % ve == 0 && pr.ldu % ve == 0)
                            : ((uintptr_t)X % 16 == 0 && ldx % 8 == 0);
#define RESQ_RF(F, M, V, P) launch_timed(residual_frag_kernel<F, M, V, P>, grid, dim3(256), 0u, s, X, m, d, ldx, nkb, qx_codes, (uint8_t*)qx_scales, qr_codes, (uint8_t*)qr_scales, partials, ehist, nm_keep, pr, bkeys)
#define RESQ_RF_MODE(F, V, P)                                        \
    switch (mode) {                                                  \
      case kResidNone: RESQ_RF(F, kResidNone, V, P); break;          \
      case kResidIdentity: RESQ_RF(F, kResidIdentity, V, P); break;  \
      case kResidDense: RESQ_RF(F, kResidDense, V, P); break;        \
      case kResidNM8: RESQ_RF(F, kResidNM8, V, P); break;            \
      case kResidNM4: RESQ_RF(F, kResidNM4, V, P); break;            \
      default: RESQ_RF(F, kResid24, V, P); break;                    \
    }
#define RESQ_RF_VEC(F, P) if (vec16) { RESQ_RF_MODE(F, true, P) } else { RESQ_RF_MODE(F, false, P) }
    if (prod && prod->kind == kProdRmsnorm) {
      if (fmt == kMX) { RESQ_RF_VEC(kMX, kProdRmsnorm) } else { RESQ_RF_VEC(kHI, kProdRmsnorm) }
    } else if (prod) {
      if (fmt == kMX) { RESQ_RF_VEC(kMX, kProdSwiglu) } else { RESQ_RF_VEC(kHI, kProdSwiglu) }
    } else {
      if (fmt == kMX) { RESQ_RF_VEC(kMX, 0) } else { RESQ_RF_VEC(kHI, 0) }
    }
#undef RESQ_RF_VEC
#undef RESQ_RF_MODE
#undef RESQ_RF
    return;
  }
  const dim3 grid((unsigned)((d / 4 + kThreads - 1) / kThreads), grid_rows(m));
  const bool vec = ((uintptr_t)X % 8 == 0) && (ldx % 4 == 0);
#define RESQ_RK(F, M, V) hipLaunchKernelGGL((residual_kernel<F, M, V>), grid, dim3(kThreads), 0, s, X, m, m, d, ldx, qx_codes, qx_scales, qr_codes, qr_scales, keep_mask, partials, nm_keep)
#define RESQ_RK_MODE(F, V)                                       \
  switch (mode) {                                                \
    case kResidNone: RESQ_RK(F, kResidNone, V); break;           \
    case kResidIdentity: RESQ_RK(F, kResidIdentity, V); break;   \
    case kResid24: RESQ_RK(F, kResid24, V); break;               \
    case kResidNM4: RESQ_RK(F, kResidNM4, V); break;             \
    case kResidNM8: RESQ_RK(F, kResidNM8, V); break;             \
    default: RESQ_RK(F, kResidDense, V); break;                  \
  }
  if (fmt == kMX) { if (vec) { RESQ_RK_MODE(kMX, true) } else { RESQ_RK_MODE(kMX, false) } }
  else { if (vec) { RESQ_RK_MODE(kHI, true) } else { RESQ_RK_MODE(kHI, false) } }
#undef RESQ_RK_MODE
#undef RESQ_RK
}

}  // namespace resq
