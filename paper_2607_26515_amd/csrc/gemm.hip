// FP4 GEMM on gfx950 scaled MFMA (v_mfma_scale_f32_32x32x64_f8f6f4):
//     Y[M][N] = Q(X) Q(W)^T  (+ S(Q(dX)) Q(W)^T into the same accumulators)   (Eq. 1, Eq. 4)
//
// MFMA operand layout (32x32x64): lane l holds row (A) / column (B) l%32 and the 32
// consecutive K elements (l/32)*32 .. +31 of the 64-wide K step, packed 4 bits (FP4) or 6
// bits (FP6) per element from bit 0 upwards; its E8M0 scale covers those 32 elements.
// Accumulator register r of lane l is row 8*(r/4) + 4*(l/32) + r%4, column l%32.
//
// MXFP4 maps directly: E2M1 codes and E8M0 scales are the MFMA's own formats.
// HiF4: the level-1 scale s1 = 2^e (1 + m/4) is not a power of two, so no FP4/FP6 operand
// can carry it.  The activation value V 2^(e-37) (V <= 196) is split into two exact E2M3
// operands (hi, lo) and the weight element k 2^-b into an exact BF6 E3M2 operand with E8M0
// 2^(e_w - 35); the remaining weight factor (4 + m_w) is constant per output column, i.e. per
// lane, and is applied once per 64-K step: acc += (4 + m_w) * P_step.
#include "kernels.h"
#include "device_fp4.h"

namespace resq {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

struct GemmParams {
  int64_t M, N, K;
  const uint8_t* a_codes[2];
  const uint8_t* a_scales[2];
  const uint8_t* a_frag[2];
  const uint8_t* a_c1[2];
  int n_terms;
  const uint8_t* blockmask;
  const uint8_t* b_codes;
  const void* b_scales;
  float* Y;
  int64_t ldy;
};

template <int FA, int FB>
__device__ __forceinline__ v16f mfma(const v8i& a, const v8i& b, const v16f& c, int sa, int sb) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, FA, FB, 0, sa, 0, sb);
}

__device__ __forceinline__ v8i zero_v8i() {
  v8i z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = 0;
  return z;
}

// Decode one lane's 32 HiF4 weight codes into packed BF6 E3M2 (6 dwords).
__device__ __forceinline__ v8i decode_w_e3m2(uint4 cw, uint32_t meta, int half) {
  const uint32_t words[4] = {cw.x, cw.y, cw.z, cw.w};
  uint32_t out[6] = {0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const uint32_t code = (words[i >> 3] >> (4 * (i & 7))) & 15u;
    const int h = half * 8 + (i >> 2);
    const int b = (int)((meta >> (8 + (h >> 1))) & 1u) + (int)((meta >> (16 + h)) & 1u);
    const uint32_t f = hif4_e3m2(code, b);
    const int bit = 6 * i;
    out[bit >> 5] |= f << (bit & 31);
    if ((bit & 31) > 26) out[(bit >> 5) + 1] |= f >> (32 - (bit & 31));
  }
  v8i r = zero_v8i();
#pragma unroll
  for (int w = 0; w < 6; ++w) r[w] = (int)out[w];
  return r;
}

template <int FMT, int TM, int TN, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN) void gemm_kernel(GemmParams p) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int64_t m0 = ((int64_t)blockIdx.y * WM + wm) * TM * 32;
  const int64_t n0 = ((int64_t)blockIdx.x * WN + wn) * TN * 32;
  // MXFP4 allows K % 64 == 32: the last step then has only its first 32-element half
  const int64_t nkb = (p.K + 63) / 64;
  const int64_t row_tiles = (p.M + 31) / 32;
  const int half = lane >> 5;
  const int l32 = lane & 31;

  v16f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  for (int64_t kb = 0; kb < nkb; ++kb) {
    // ---- B fragments (Q(W)) ----
    v8i bf[TN];
    int sb[TN];
    float fb[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int64_t col = n0 + j * 32 + l32;
      const bool kin = kb * 64 + half * 32 < p.K;  // false only in an MXFP4 half step
      const bool ok = col < p.N && kin;
      const int64_t cc = col < p.N ? col : 0;
      const int64_t ko = kin ? kb * 32 + half * 16 : 0;
      const uint4 cw = *reinterpret_cast<const uint4*>(p.b_codes + cc * (p.K / 2) + ko);
      if constexpr (FMT == 0) {
        bf[j] = zero_v8i();
        bf[j][0] = ok ? (int)cw.x : 0; bf[j][1] = ok ? (int)cw.y : 0;
        bf[j][2] = ok ? (int)cw.z : 0; bf[j][3] = ok ? (int)cw.w : 0;
        sb[j] = reinterpret_cast<const uint8_t*>(p.b_scales)[cc * (p.K / 32) + (kin ? kb * 2 + half : 0)];
        fb[j] = 1.f;
      } else {
        const uint32_t mt = reinterpret_cast<const uint32_t*>(p.b_scales)[cc * nkb + kb];
        bf[j] = ok ? decode_w_e3m2(cw, mt, half) : zero_v8i();
        sb[j] = (int)((mt & 0xFFu) >> 2) + 92;
        fb[j] = ok ? (float)(4 + (mt & 3u)) : 0.f;
      }
    }
    // ---- A fragments and MFMAs ----
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int64_t t = m0 / 32 + i;
      if (t >= row_tiles) continue;  // wave-uniform
      const bool resid = p.n_terms > 1 &&
                         (p.blockmask == nullptr || ((p.blockmask[(t * nkb + kb) >> 3] >> ((t * nkb + kb) & 7)) & 1));
      if constexpr (FMT == 0) {
        const int64_t row = t * 32 + l32;
        const bool kin = kb * 64 + half * 32 < p.K;
        const bool ok = row < p.M && kin;
        const int64_t rr = row < p.M ? row : 0;
        const int64_t ko = kin ? kb * 32 + half * 16 : 0;
        const int64_t so = kin ? kb * 2 + half : 0;
        v8i ax = zero_v8i(), ar = zero_v8i();
        const uint4 cx = *reinterpret_cast<const uint4*>(p.a_codes[0] + rr * (p.K / 2) + ko);
        const int sx = p.a_scales[0][rr * (p.K / 32) + so];
        if (ok) { ax[0] = (int)cx.x; ax[1] = (int)cx.y; ax[2] = (int)cx.z; ax[3] = (int)cx.w; }
        int sr = 127;
        if (resid) {
          const uint4 cr = *reinterpret_cast<const uint4*>(p.a_codes[1] + rr * (p.K / 2) + ko);
          sr = p.a_scales[1][rr * (p.K / 32) + so];
          if (ok) { ar[0] = (int)cr.x; ar[1] = (int)cr.y; ar[2] = (int)cr.z; ar[3] = (int)cr.w; }
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          acc[i][j] = mfma<4, 4>(ax, bf[j], acc[i][j], sx, sb[j]);
          if (resid) acc[i][j] = mfma<4, 4>(ar, bf[j], acc[i][j], sr, sb[j]);
        }
      } else {
        const int64_t fbase = (t * nkb + kb);
        v8i xh = zero_v8i(), xl = zero_v8i(), rh = zero_v8i(), rl = zero_v8i();
        {
          const uint32_t* ph = reinterpret_cast<const uint32_t*>(p.a_frag[0] + ((fbase * 2 + 0) * 64 + lane) * 24);
          const uint32_t* pl = reinterpret_cast<const uint32_t*>(p.a_frag[0] + ((fbase * 2 + 1) * 64 + lane) * 24);
#pragma unroll
          for (int w = 0; w < 6; ++w) { xh[w] = (int)ph[w]; xl[w] = (int)pl[w]; }
        }
        const int ex = p.a_c1[0][fbase * 64 + lane] >> 2;
        int er = 0;
        if (resid) {
          const uint32_t* ph = reinterpret_cast<const uint32_t*>(p.a_frag[1] + ((fbase * 2 + 0) * 64 + lane) * 24);
          const uint32_t* pl = reinterpret_cast<const uint32_t*>(p.a_frag[1] + ((fbase * 2 + 1) * 64 + lane) * 24);
#pragma unroll
          for (int w = 0; w < 6; ++w) { rh[w] = (int)ph[w]; rl[w] = (int)pl[w]; }
          er = p.a_c1[1][fbase * 64 + lane] >> 2;
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          v16f P;
#pragma unroll
          for (int r = 0; r < 16; ++r) P[r] = 0.f;
          P = mfma<2, 3>(xh, bf[j], P, ex + 97, sb[j]);
          P = mfma<2, 3>(xl, bf[j], P, ex + 93, sb[j]);
          if (resid) {
            P = mfma<2, 3>(rh, bf[j], P, er + 97, sb[j]);
            P = mfma<2, 3>(rl, bf[j], P, er + 93, sb[j]);
          }
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] = fmaf(P[r], fb[j], acc[i][j][r]);
        }
      }
    }
  }
  // ---- epilogue ----
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int64_t col = n0 + j * 32 + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + i * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (row < p.M && col < p.N) p.Y[row * p.ldy + col] = acc[i][j][r];
      }
    }
}

template <int FMT, int TM, int TN, int WM, int WN>
void launch_cfg(const GemmParams& p, hipStream_t s) {
  const int64_t bm = WM * TM * 32, bn = WN * TN * 32;
  const dim3 grid((unsigned)((p.N + bn - 1) / bn), (unsigned)((p.M + bm - 1) / bm));
  hipLaunchKernelGGL((gemm_kernel<FMT, TM, TN, WM, WN>), grid, dim3(64 * WM * WN), 0, s, p);
}

}  // namespace

void launch_gemm(const GemmOperands& op, hipStream_t s) {
  if (op.M == 0 || op.N == 0) return;
  GemmParams p;
  p.M = op.M; p.N = op.N; p.K = op.K;
  for (int t = 0; t < 2; ++t) {
    p.a_codes[t] = op.a_codes[t]; p.a_scales[t] = op.a_scales[t];
    p.a_frag[t] = op.a_frag[t]; p.a_c1[t] = op.a_c1[t];
  }
  p.n_terms = op.n_terms;
  p.blockmask = op.blockmask;
  p.b_codes = op.b_codes; p.b_scales = op.b_scales;
  p.Y = op.Y; p.ldy = op.ldy;
  // tile choice: prefer large tiles while keeping >= 256 workgroups in flight
  const int64_t wg_128x128 = ((op.N + 127) / 128) * ((op.M + 127) / 128);
  const int64_t wg_64x64 = ((op.N + 63) / 64) * ((op.M + 63) / 64);
  if (op.fmt == 0) {
    if (wg_128x128 >= 256) launch_cfg<0, 2, 2, 2, 2>(p, s);
    else if (wg_64x64 >= 256) launch_cfg<0, 1, 1, 2, 2>(p, s);
    else launch_cfg<0, 1, 1, 1, 1>(p, s);
  } else {
    if (wg_128x128 >= 256) launch_cfg<1, 2, 2, 2, 2>(p, s);
    else if (wg_64x64 >= 256) launch_cfg<1, 1, 1, 2, 2>(p, s);
    else launch_cfg<1, 1, 1, 1, 1>(p, s);
  }
}

}  // namespace resq
