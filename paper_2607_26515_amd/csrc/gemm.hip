// FP4 GEMM on gfx950 scaled MFMA (v_mfma_scale_f32_32x32x64_f8f6f4):
//     Y[M][N] = Q(X) Q(W)^T  (+ S(Q(dX)) Q(W)^T into the same accumulators)   (Eq. 1, Eq. 4)
//
// MFMA operand layout (32x32x64): lane l holds row (A) / column (B) l%32 and the 32
// consecutive K elements (l/32)*32 .. +31 of the 64-wide K step, packed 4 bits (FP4) or 6
// bits (FP6) per element from bit 0 upwards; its E8M0 scale covers those 32 elements.
// Accumulator register r of lane l is row 8*(r/4) + 4*(l/32) + r%4, column l%32.
// Operands arrive "fragment-major" (pack.hip): a wave loads one fragment as one contiguous
// block of 64 lane records.
//
// MXFP4 maps directly: E2M1 codes and E8M0 scales are the MFMA's own formats.
// HiF4: the level-1 scale s1 = 2^e (1 + m/4) is not a power of two, so no FP4/FP6 operand
// can carry it.  The activation value V 2^(e-37) (V <= 196) is split into two exact E2M3
// operands (hi, lo) and the weight element k 2^-b is an exact BF6 E3M2 operand with E8M0
// 2^(e_w - 35); the remaining weight factor (4 + m_w) is constant per output column, i.e. per
// lane, and is applied once per 64-K step: acc += (4 + m_w) * P_step.
//
// Work split: a workgroup owns a (WM*TM*32) x (WN*TN*32) output tile; its waves split it
// WM x WN and split K WK ways (interleaved K steps).  The WK partial accumulators are summed
// through LDS in a fixed order, so results do not depend on timing.  Workgroups are mapped
// to tiles in contiguous chunks per XCD (workgroup b runs on XCD b % 8), so tiles that share
// a weight column block run on the same XCD and share its L2.
#include "kernels.h"
#include "device_fp4.h"
#include "gemm_lds.h"

namespace resq {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kXcds = 8;

struct GemmParams {
  int64_t M, N, K, nkb, mt_tiles, nt_tiles;
  const uint8_t* a_frag[2];
  const uint8_t* a_sc[2];
  uint32_t a_frag_bytes, a_sc_bytes, b_frag_bytes, b_sc_bytes, mask_bytes;
  const uint8_t* blockmask;
  const uint8_t* b_frag;
  const uint8_t* b_sc;
  float* Y;
  int64_t ldy;
  int64_t grid_m, grid_n, per_xcd;
};

template <int FA, int FB>
__device__ __forceinline__ v16f mfma(const v8i& a, const v8i& b, const v16f& c, int sa, int sb) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, FA, FB, 0, sa, 0, sb);
}

// Per-stage register fragments of one wave.
template <int FMT, int TM, int TN, int NT>
struct Stage {
  // MXFP4: 1 uint4 per fragment; HiF4 A: 3 uint4 (hi | lo), HiF4 B: 3 uint2 (24 B)
  uint4 a[NT][TM][FMT == 0 ? 1 : 3];
  uint32_t sa[NT][TM];
  uint4 b[TN][FMT == 0 ? 1 : 2];  // HiF4 B: 24 B held in 1.5 uint4 (second half-used)
  uint32_t sb[TN];
  uint32_t keep[TM];  // 32x64 block-skip: kept bit of the residual block (BS only)
};

// Loads one K step's fragments.  Every load is issued unconditionally (indices clamped to
// valid fragments; the compute step skips the tiles past the edge), so the compiler can count
// outstanding loads exactly and keep STAGES-1 K steps in flight.
template <int FMT, int TM, int TN, int NT, bool BS>
__device__ __forceinline__ void load_stage(Stage<FMT, TM, TN, NT>& s, const GemmParams& p,
                                           int64_t t0, int64_t tn0, int64_t kb, int lane) {
  const int64_t kc = kb < p.nkb ? kb : p.nkb - 1;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int64_t tn = (tn0 + j) < p.nt_tiles ? (tn0 + j) : p.nt_tiles - 1;
    const int64_t f = (tn * p.nkb + kc) * 64 + lane;
    if constexpr (FMT == 0) {
      s.b[j][0] = *reinterpret_cast<const uint4*>(p.b_frag + f * 16);
    } else {
      const uint2* q = reinterpret_cast<const uint2*>(p.b_frag + f * 24);
      const uint2 x0 = q[0], x1 = q[1], x2 = q[2];
      s.b[j][0] = make_uint4(x0.x, x0.y, x1.x, x1.y);
      s.b[j][1] = make_uint4(x2.x, x2.y, 0u, 0u);
    }
    s.sb[j] = p.b_sc[f];
  }
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int64_t tm = (t0 + i) < p.mt_tiles ? (t0 + i) : p.mt_tiles - 1;
      const int64_t f = (tm * p.nkb + kc) * 64 + lane;
      if constexpr (FMT == 0) {
        s.a[t][i][0] = *reinterpret_cast<const uint4*>(p.a_frag[t] + f * 16);
      } else {
        const uint4* q = reinterpret_cast<const uint4*>(p.a_frag[t] + f * 48);
        s.a[t][i][0] = q[0];
        s.a[t][i][1] = q[1];
        s.a[t][i][2] = q[2];
      }
      s.sa[t][i] = p.a_sc[t][f];
    }
  if constexpr (BS) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int64_t tm = (t0 + i) < p.mt_tiles ? (t0 + i) : p.mt_tiles - 1;
      const int64_t bit = tm * p.nkb + kc;
      s.keep[i] = p.blockmask[bit >> 3] >> (bit & 7);
    }
  }
}

__device__ __forceinline__ v8i v8_from(uint4 a, uint4 b) {
  v8i r;
  r[0] = (int)a.x; r[1] = (int)a.y; r[2] = (int)a.z; r[3] = (int)a.w;
  r[4] = (int)b.x; r[5] = (int)b.y; r[6] = (int)b.z; r[7] = (int)b.w;
  return r;
}

template <int FMT, int TM, int TN, int NT, bool BS>
__device__ __forceinline__ void compute_stage(const Stage<FMT, TM, TN, NT>& s, const GemmParams& p,
                                              int64_t t0, int64_t tn0, v16f (&acc)[TM][TN]) {
  const uint4 z = make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int64_t tm = t0 + i;
    if (tm >= p.mt_tiles) continue;  // wave-uniform
    bool res = NT > 1;
    if constexpr (BS) res = (__builtin_amdgcn_readfirstlane(s.keep[i]) & 1u) != 0;  // wave-uniform
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      if (tn0 + j >= p.nt_tiles) continue;  // wave-uniform
      if constexpr (FMT == 0) {
        const v8i b = v8_from(s.b[j][0], z);
        acc[i][j] = mfma<4, 4>(v8_from(s.a[0][i][0], z), b, acc[i][j], (int)s.sa[0][i], (int)s.sb[j]);
        if (NT > 1 && res)
          acc[i][j] = mfma<4, 4>(v8_from(s.a[NT - 1][i][0], z), b, acc[i][j], (int)s.sa[NT - 1][i], (int)s.sb[j]);
      } else {
        const v8i b = v8_from(s.b[j][0], s.b[j][1]);
        const int sb = (int)(s.sb[j] >> 2) + 92;
        const float fb = (float)(4 + (s.sb[j] & 3u));
        // E2M3 hi = dwords 0-5 of the 48-byte lane record, lo = dwords 6-11
        const uint4* a0 = s.a[0][i];
        const v8i xh = v8_from(a0[0], make_uint4(a0[1].x, a0[1].y, 0u, 0u));
        const v8i xl = v8_from(make_uint4(a0[1].z, a0[1].w, a0[2].x, a0[2].y), make_uint4(a0[2].z, a0[2].w, 0u, 0u));
        const int ex = (int)(s.sa[0][i] >> 2);
        v16f P;
#pragma unroll
        for (int r = 0; r < 16; ++r) P[r] = 0.f;
        P = mfma<2, 3>(xh, b, P, ex + 97, sb);
        P = mfma<2, 3>(xl, b, P, ex + 93, sb);
        if (NT > 1 && res) {
          const uint4* a1 = s.a[NT - 1][i];
          const v8i rh = v8_from(a1[0], make_uint4(a1[1].x, a1[1].y, 0u, 0u));
          const v8i rl = v8_from(make_uint4(a1[1].z, a1[1].w, a1[2].x, a1[2].y), make_uint4(a1[2].z, a1[2].w, 0u, 0u));
          const int er = (int)(s.sa[NT - 1][i] >> 2);
          P = mfma<2, 3>(rh, b, P, er + 97, sb);
          P = mfma<2, 3>(rl, b, P, er + 93, sb);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = fmaf(P[r], fb, acc[i][j][r]);
      }
    }
  }
}

template <int FMT, int TM, int TN, int WM, int WN, int WK, int NT, int STAGES, bool BS>
__global__ __launch_bounds__(64 * WM * WN * WK) void gemm_kernel(GemmParams p) {
  extern __shared__ float red[];
  // XCD-chunked tile order: workgroup b runs on XCD b % 8 and takes the (b / 8)-th tile of
  // that XCD's contiguous chunk; tiles are numbered row-tile fastest.
  const int64_t b = blockIdx.x;
  const int64_t tile = (b % kXcds) * p.per_xcd + b / kXcds;
  if (tile >= p.grid_m * p.grid_n) return;
  const int64_t wg_m = tile % p.grid_m, wg_n = tile / p.grid_m;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave % WM, wn = (wave / WM) % WN, wk = wave / (WM * WN);
  const int64_t t0 = (wg_m * WM + wm) * TM;   // first row tile of this wave
  const int64_t tn0 = (wg_n * WN + wn) * TN;  // first column tile

  v16f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // software pipeline over this wave's K steps wk, wk + WK, ...: STAGES-1 steps in flight
  const int64_t n_it = p.nkb > wk ? (p.nkb - wk + WK - 1) / WK : 0;
  if (n_it > 0) {
    Stage<FMT, TM, TN, NT> st[STAGES];
#pragma unroll
    for (int sidx = 0; sidx < STAGES - 1; ++sidx)
      load_stage<FMT, TM, TN, NT, BS>(st[sidx], p, t0, tn0, wk + (int64_t)sidx * WK, lane);
    for (int64_t it = 0; it < n_it; it += STAGES) {
#pragma unroll
      for (int sidx = 0; sidx < STAGES; ++sidx) {
        load_stage<FMT, TM, TN, NT, BS>(st[(sidx + STAGES - 1) % STAGES], p, t0, tn0,
                                        wk + (it + sidx + STAGES - 1) * WK, lane);
        if (it + sidx < n_it) compute_stage<FMT, TM, TN, NT, BS>(st[sidx], p, t0, tn0, acc);
      }
    }
  }

  if constexpr (WK > 1) {
    // fixed-order reduction of the K-split partial sums through LDS
    constexpr int R = TM * TN * 16;
    const int wmn = wave % (WM * WN);
    if (wk > 0) {
      float* dst = red + ((size_t)((wk - 1) * WM * WN + wmn) * R) * 64;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) dst[((i * TN + j) * 16 + r) * 64 + lane] = acc[i][j][r];
    }
    __syncthreads();
    if (wk > 0) return;
#pragma unroll
    for (int q = 1; q < WK; ++q) {
      const float* src = red + ((size_t)((q - 1) * WM * WN + wmn) * R) * 64;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] += src[((i * TN + j) * 16 + r) * 64 + lane];
    }
  }

  const int half = lane >> 5, l32 = lane & 31;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int64_t col = (tn0 + j) * 32 + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = (t0 + i) * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (row < p.M && col < p.N) p.Y[row * p.ldy + col] = acc[i][j][r];
      }
    }
}

// ---------------------------------------------------------------------------------------
// LDS-shared main loop (gemm_lds.h): cooperative per-workgroup operand fetch
// ---------------------------------------------------------------------------------------
template <int FMT, int WM, int WN, int TM, int TN, int NT, int R, bool BS>
__global__ __launch_bounds__(64 * WM * WN) void gemm_lds_kernel(GemmParams p) {
  using G = lds::Geo<FMT, WM, WN, TM, TN, NT>;
  using lds::v4i;
  using lds::v2i;
  extern __shared__ __attribute__((aligned(256))) uint8_t smem[];
  constexpr int MASK_OFF = G::SB_OFF + G::NTW * 64;
  constexpr int STAGE = (MASK_OFF + 64 + 255) / 256 * 256;
  constexpr uint32_t BAD = 0xFFFFFFF0u;  // an offset past every operand: the load returns 0

  const int64_t b = blockIdx.x;
  const int64_t tile = (b % kXcds) * p.per_xcd + b / kXcds;
  if (tile >= p.grid_m * p.grid_n) return;
  const int64_t wg_m = tile % p.grid_m, wg_n = tile / p.grid_m;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int wm = wave % WM, wn = wave / WM;
  const uint32_t T0 = (uint32_t)(wg_m * G::MTW), N0 = (uint32_t)(wg_n * G::NTW);
  const uint32_t nkb = (uint32_t)p.nkb;

  __amdgpu_buffer_rsrc_t ra[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) ra[t] = lds::make_rsrc(p.a_frag[t], p.a_frag_bytes);
  const __amdgpu_buffer_rsrc_t rb = lds::make_rsrc(p.b_frag, p.b_frag_bytes);
  // scale / mask loads: wave w < NT fetches A term w's scales, wave NT the B scales and
  // wave NT + 1 the block-skip mask words; other waves issue an out-of-range (zero) load
  const __amdgpu_buffer_rsrc_t rs =
      wave < NT ? lds::make_rsrc(p.a_sc[wave < NT ? wave : 0], p.a_sc_bytes)
                : (wave == NT ? lds::make_rsrc(p.b_sc, p.b_sc_bytes)
                              : lds::make_rsrc(p.blockmask, BS ? p.mask_bytes : 0u));

  // per-thread load offsets at kb = 0 (advanced by kb * step each K step) and LDS offsets
  constexpr uint32_t A_STEP = 64 * G::FA, B_STEP = 64 * G::FB;
  uint32_t a_off[G::A_PER], a_lds[G::A_PER];
  bool a_ok[G::A_PER];
#pragma unroll
  for (int i = 0; i < G::A_PER; ++i) {
    const uint32_t c = (uint32_t)(tid + i * G::kThreads);
    a_ok[i] = c < (uint32_t)G::A_CHUNKS;
    if constexpr (FMT == 0) {
      a_off[i] = ((T0 + c / 64) * nkb * 64 + c % 64) * 16;
      a_lds[i] = c * 16;
    } else {
      const uint32_t w = c % 192;
      a_off[i] = ((T0 + c / 192) * nkb * 64 + w / 3) * 48 + (w % 3) * 16;
      a_lds[i] = (c / 192) * 3072 + (w % 3) * 1024 + (w / 3) * 16;
    }
  }
  uint32_t b_off[G::B_PER], b_lds[G::B_PER];
  bool b_ok[G::B_PER];
#pragma unroll
  for (int i = 0; i < G::B_PER; ++i) {
    const uint32_t c = (uint32_t)(tid + i * G::kThreads);
    b_ok[i] = c < (uint32_t)G::B_CHUNKS;
    if constexpr (FMT == 0) {
      b_off[i] = ((N0 + c / 64) * nkb * 64 + c % 64) * 16;
      b_lds[i] = G::A_BYTES + c * 16;
    } else {
      const uint32_t w = c % 192, r = w / 3, q = w % 3;
      b_off[i] = ((N0 + c / 192) * nkb * 64 + r) * 24 + q * 8;
      const uint32_t base = G::A_BYTES + (c / 192) * 1536;
      b_lds[i] = q < 2 ? base + r * 16 + q * 8 : base + 1024 + r * 8;
    }
  }
  bool s_ok = false;
  uint32_t s_off = 0, s_lds = 0;
  if (wave < NT) {
    s_ok = lane < G::MTW * 16;
    s_off = (T0 + lane / 16) * nkb * 64 + (lane % 16) * 4;
    s_lds = G::SA_OFF + wave * G::MTW * 64 + lane * 4;
  } else if (wave == NT) {
    s_ok = lane < G::NTW * 16;
    s_off = (N0 + lane / 16) * nkb * 64 + (lane % 16) * 4;
    s_lds = G::SB_OFF + lane * 4;
  } else if (BS && wave == NT + 1) {
    s_ok = lane < G::MTW;
    s_lds = MASK_OFF + lane * 4;
  }

  v4i ar[R][NT][G::A_PER];
  v4i br4[R][FMT == 0 ? G::B_PER : 1];
  v2i br2[R][FMT == 0 ? 1 : G::B_PER];
  int sr[R];

  auto issue = [&](int s, uint32_t kb) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < G::A_PER; ++i)
        ar[s][t][i] = lds::ld16(ra[t], a_ok[i] ? a_off[i] + kb * A_STEP : BAD);
#pragma unroll
    for (int i = 0; i < G::B_PER; ++i) {
      if constexpr (FMT == 0) br4[s][i] = lds::ld16(rb, b_ok[i] ? b_off[i] + kb * B_STEP : BAD);
      else br2[s][i] = lds::ld8(rb, b_ok[i] ? b_off[i] + kb * B_STEP : BAD);
    }
    uint32_t so = BAD;
    if (s_ok) so = (BS && wave == NT + 1) ? (((T0 + lane) * nkb + kb) >> 5) * 4 : s_off + kb * 64;
    sr[s] = lds::ld4(rs, so);
  };

  auto store = [&](int s, int buf, uint32_t kb) {
    uint8_t* st = smem + buf * STAGE;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < G::A_PER; ++i)
        if (a_ok[i]) *reinterpret_cast<v4i*>(st + t * G::MTW * G::A_FRAG + a_lds[i]) = ar[s][t][i];
#pragma unroll
    for (int i = 0; i < G::B_PER; ++i)
      if (b_ok[i]) {
        if constexpr (FMT == 0) *reinterpret_cast<v4i*>(st + b_lds[i]) = br4[s][i];
        else *reinterpret_cast<v2i*>(st + b_lds[i]) = br2[s][i];
      }
    if (s_ok) {
      int v = sr[s];
      if (BS && wave == NT + 1) v = (v >> (((T0 + lane) * nkb + kb) & 31)) & 1;
      *reinterpret_cast<int*>(st + s_lds) = v;
    }
  };

  v16f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // One K step's MFMA operands of this wave, read from an LDS stage.  Two register sets
  // alternate: step k+1's operands are read while step k's MFMAs run.
  struct Frag {
    v8i b[TN];
    int sb[TN];
    v8i a[NT][TM][FMT == 0 ? 1 : 2];  // HiF4: E2M3 hi, lo
    int sa[NT][TM];
    int keep[TM];
  };
  Frag F[2];

  auto read = [&](Frag& f, int buf) {
    const uint8_t* st = smem + buf * STAGE;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int lj = wn * TN + j;
      if constexpr (FMT == 0) {
        const v4i x = *reinterpret_cast<const v4i*>(st + G::A_BYTES + lj * 1024 + lane * 16);
        f.b[j] = v8i{x[0], x[1], x[2], x[3], 0, 0, 0, 0};
      } else {
        const uint8_t* bb = st + G::A_BYTES + lj * 1536;
        const v4i x = *reinterpret_cast<const v4i*>(bb + lane * 16);
        const v2i y = *reinterpret_cast<const v2i*>(bb + 1024 + lane * 8);
        f.b[j] = v8i{x[0], x[1], x[2], x[3], y[0], y[1], 0, 0};
      }
      f.sb[j] = st[G::SB_OFF + lj * 64 + lane];
    }
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int li = t * G::MTW + wm * TM + i;
        if constexpr (FMT == 0) {
          const v4i x = *reinterpret_cast<const v4i*>(st + li * 1024 + lane * 16);
          f.a[t][i][0] = v8i{x[0], x[1], x[2], x[3], 0, 0, 0, 0};
        } else {
          const uint8_t* a0 = st + li * 3072;
          const v4i p0 = *reinterpret_cast<const v4i*>(a0 + lane * 16);
          const v4i p1 = *reinterpret_cast<const v4i*>(a0 + 1024 + lane * 16);
          const v4i p2 = *reinterpret_cast<const v4i*>(a0 + 2048 + lane * 16);
          f.a[t][i][0] = v8i{p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], 0, 0};
          f.a[t][i][1] = v8i{p1[2], p1[3], p2[0], p2[1], p2[2], p2[3], 0, 0};
        }
        f.sa[t][i] = st[G::SA_OFF + li * 64 + lane];
      }
#pragma unroll
    for (int i = 0; i < TM; ++i)
      f.keep[i] = BS ? *reinterpret_cast<const int*>(st + MASK_OFF + (wm * TM + i) * 4) : 1;
  };

  // Tiles past the edge of the output hold zero operands, so they are computed like the
  // others (their results are never stored) and the MFMAs stay branch-free.  Term-major
  // order keeps the TM x TN independent accumulator chains interleaved.
  auto mma = [&](const Frag& f) {
    bool res[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) res[i] = NT > 1 && (!BS || __builtin_amdgcn_readfirstlane(f.keep[i]) != 0);
    if constexpr (FMT == 0) {
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          if (t > 0 && !res[i]) continue;  // wave-uniform (32x64 block skip)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = mfma<4, 4>(f.a[t][i][0], f.b[j], acc[i][j], f.sa[t][i], f.sb[j]);
        }
    } else {
      v16f P[TM][TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) P[i][j][r] = 0.f;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            if (t > 0 && !res[i]) continue;  // wave-uniform (32x64 block skip)
            const int sa = (f.sa[t][i] >> 2) + (h == 0 ? 97 : 93);
#pragma unroll
            for (int j = 0; j < TN; ++j)
              P[i][j] = mfma<2, 3>(f.a[t][i][h], f.b[j], P[i][j], sa, (f.sb[j] >> 2) + 92);
          }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const float fb = (float)(4 + (f.sb[j] & 3));
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] = fmaf(P[i][j][r], fb, acc[i][j][r]);
        }
    }
  };

  // Pipeline: global loads run R stages ahead in registers; LDS holds 3 stages.  At step k
  // the waves read stage k+1 from LDS while the MFMAs of stage k run, then write stage k+2
  // into the slot that held stage k-1 and pass one barrier.  U = 6 unrolls every ring index.
  constexpr int U = 6;
  static_assert(U % R == 0, "register ring depth must divide the unroll");
  const int64_t nk = p.nkb;
  if (nk > 0) {
#pragma unroll
    for (int s = 0; s < R; ++s) issue(s, (uint32_t)s);
    store(0, 0, 0u);
    issue(0, (uint32_t)R);
    if (nk > 1) store(1 % R, 1, 1u);
    issue(1 % R, (uint32_t)(R + 1));
    __syncthreads();
    read(F[0], 0);
    for (int64_t k0 = 0; k0 < nk; k0 += U) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t k = k0 + u;
        if (k < nk) {
          if (k + 1 < nk) read(F[(u + 1) & 1], (int)((k + 1) % 3));
          mma(F[u & 1]);
          if (k + 2 < nk) store((u + 2) % R, (int)((k + 2) % 3), (uint32_t)(k + 2));
        }
        issue((u + 2) % R, (uint32_t)(k + 2 + R));
        if (k < nk) __syncthreads();
      }
    }
  }

  const int half = lane >> 5, l32 = lane & 31;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int64_t col = ((int64_t)N0 + wn * TN + j) * 32 + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = ((int64_t)T0 + wm * TM + i) * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (row < p.M && col < p.N) p.Y[row * p.ldy + col] = acc[i][j][r];
      }
    }
}

template <int FMT, int WM, int WN, int TM, int TN, int R>
void launch_lds(GemmParams p, int n_terms, hipStream_t s) {
  p.grid_m = (p.mt_tiles + WM * TM - 1) / (WM * TM);
  p.grid_n = (p.nt_tiles + WN * TN - 1) / (WN * TN);
  const int64_t tiles = p.grid_m * p.grid_n;
  p.per_xcd = (tiles + kXcds - 1) / kXcds;
  const dim3 grid((unsigned)(p.per_xcd * kXcds));
  const dim3 block(64 * WM * WN);
  auto lds_bytes = [](int nt) {
    const int a = nt * WM * TM * 64 * (FMT == 0 ? 16 : 48);
    const int b = WN * TN * 64 * (FMT == 0 ? 16 : 24);
    const int mask_off = a + b + nt * WM * TM * 64 + WN * TN * 64;
    return (size_t)3 * ((mask_off + 64 + 255) / 256 * 256);
  };
  if (n_terms > 1 && p.blockmask != nullptr)
    hipLaunchKernelGGL((gemm_lds_kernel<FMT, WM, WN, TM, TN, 2, R, true>), grid, block, lds_bytes(2), s, p);
  else if (n_terms > 1)
    hipLaunchKernelGGL((gemm_lds_kernel<FMT, WM, WN, TM, TN, 2, R, false>), grid, block, lds_bytes(2), s, p);
  else
    hipLaunchKernelGGL((gemm_lds_kernel<FMT, WM, WN, TM, TN, 1, R, false>), grid, block, lds_bytes(1), s, p);
}

template <int FMT, int TM, int TN, int WM, int WN, int WK, int STAGES>
void launch_cfg(GemmParams p, int n_terms, hipStream_t s) {
  constexpr int BM = WM * TM, BN = WN * TN;  // in 32-row / 32-column tiles
  p.grid_m = (p.mt_tiles + BM - 1) / BM;
  p.grid_n = (p.nt_tiles + BN - 1) / BN;
  const int64_t tiles = p.grid_m * p.grid_n;
  p.per_xcd = (tiles + kXcds - 1) / kXcds;
  const dim3 grid((unsigned)(p.per_xcd * kXcds));
  const dim3 block(64 * WM * WN * WK);
  const size_t lds = WK > 1 ? (size_t)(WK - 1) * WM * WN * TM * TN * 16 * 64 * sizeof(float) : 0;
  if (n_terms > 1 && p.blockmask != nullptr)
    hipLaunchKernelGGL((gemm_kernel<FMT, TM, TN, WM, WN, WK, 2, STAGES, true>), grid, block, lds, s, p);
  else if (n_terms > 1)
    hipLaunchKernelGGL((gemm_kernel<FMT, TM, TN, WM, WN, WK, 2, STAGES, false>), grid, block, lds, s, p);
  else
    hipLaunchKernelGGL((gemm_kernel<FMT, TM, TN, WM, WN, WK, 1, STAGES, false>), grid, block, lds, s, p);
}

template <int FMT>
void launch_fmt(const GemmParams& p, int n_terms, hipStream_t s) {
  auto wgs = [&](int bm, int bn) { return ((p.mt_tiles + bm - 1) / bm) * ((p.nt_tiles + bn - 1) / bn); };
  // Prefer the largest tile that still yields about one workgroup per CU; small outputs
  // split K across the four waves of a workgroup instead.
  // Register-ring depth: enough K steps in flight to cover HBM latency on the weight stream
  // (HiF4 fragments are larger, so its ring is shallower).
  constexpr int SL = FMT == 0 ? 5 : 3;
  constexpr int SS = FMT == 0 ? 6 : 4;
  if (wgs(4, 4) >= 240)
    launch_lds<FMT, 2, 2, 2, 2, FMT == 0 ? 6 : 2>(p, n_terms, s);
  else
    launch_lds<FMT, 2, 2, 1, 1, FMT == 0 ? 6 : 3>(p, n_terms, s);
}

}  // namespace

void launch_gemm(const GemmOperands& op, hipStream_t s) {
  if (op.M == 0 || op.N == 0) return;
  GemmParams p{};
  p.M = op.M; p.N = op.N; p.K = op.K;
  p.nkb = (op.K + 63) / 64;
  p.mt_tiles = (op.M + 31) / 32;
  p.nt_tiles = (op.N + 31) / 32;
  for (int t = 0; t < 2; ++t) { p.a_frag[t] = op.a_frag[t]; p.a_sc[t] = op.a_sc[t]; }
  p.blockmask = op.blockmask;
  p.b_frag = op.b_frag; p.b_sc = op.b_sc;
  p.Y = op.Y; p.ldy = op.ldy;
  const int amode = op.fmt == 0 ? kPackMx : kPackHiA, bmode = op.fmt == 0 ? kPackMx : kPackHiB;
  p.a_frag_bytes = (uint32_t)frag_bytes(amode, op.M, op.K);
  p.a_sc_bytes = (uint32_t)frag_scale_bytes(op.M, op.K);
  p.b_frag_bytes = (uint32_t)frag_bytes(bmode, op.N, op.K);
  p.b_sc_bytes = (uint32_t)frag_scale_bytes(op.N, op.K);
  p.mask_bytes = (uint32_t)((p.mt_tiles * p.nkb + 31) / 32 * 4);
  if (op.fmt == 0) launch_fmt<0>(p, op.n_terms, s);
  else launch_fmt<1>(p, op.n_terms, s);
}

}  // namespace resq
