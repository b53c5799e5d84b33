// Mixed-precision rollout GEMMs of the paper's precision ablation (Table 1): weight-only FP4
// (W4A16: Y = X Q(W)^T, bf16 activations) and activation-only FP4 (W16A4: Y = Q(X) W^T, bf16
// weights), float32 Y.
//
// Both run on gfx950's bf16 MFMA (v_mfma_f32_32x32x16_bf16, float32 accumulation).  Every
// FP4 value is exact in bf16 (an MXFP4 value has 2 significant bits, a HiF4 value
// k (4+m) 2^(e-35-b) at most 6), so the FP4 operand is dequantized to bf16 without rounding
// and every product is exact in float32; only the accumulation rounds.  The FP4 operand
// arrives K-major (codes + block scales, the ABI's exchange format) and is dequantized on
// its way from global memory into LDS: HBM carries 4.25 (MXFP4) or 4.5 (HiF4) bits per
// element of that operand, which is what makes W4A16 the bandwidth-saving option at decode.
//
// Data movement: a workgroup of 2 x 2 waves owns a (64 TM) x (64 TN) output tile; per K
// chunk of 64 each thread loads its share of both operands into registers (16-byte loads of
// bf16 rows or of FP4 codes), the workgroup writes them to one of two LDS buffers as bf16
// rows (K contiguous, rows padded by 16 bytes; FP4 codes dequantized on the way), and each
// wave runs TM x TN x 4 MFMAs (K = 16 each) from LDS.  Global loads run two chunks ahead of
// the MFMAs (two register stages), so each load's latency is covered by two chunks of work;
// one barrier per chunk.  Tall tiles (TM up to 4, i.e. every row of a 256-token decode batch)
// spread the dequantization of a weight chunk over more output rows; small grids with long K
// split each tile's chunks over four K groups of waves.
//
// Dequantization: MXFP4 pairs go through gfx950's scaled conversion to bf16
// (v_cvt_scalef32_pk_bf16_fp4, scale 2^E, exact); a HiF4 element is the integer k (4 + m)
// converted to float32 (exact) and scaled by 2^(e-35-b) with v_ldexp_f32 (exact), whose top
// half is its bf16 pattern.
//
// MFMA operand layout (32x32x16 bf16): lane l holds row (A) / column (B) l % 32 and the 8
// consecutive K elements 8 (l / 32) .. + 7 of the 16-wide step.  Accumulator register r of
// lane l is row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32.
#include <type_traits>

#include "kernels.h"
#include "device_fp4.h"
#include "profiler.h"

namespace resq {
namespace {

typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

constexpr int kChunk = 64;              // K elements per LDS chunk
constexpr int kRowHalves = kChunk + 8;  // bf16 per LDS row (16 bytes of padding)

struct MixedParams {
  int64_t M, N, K;
  // the bf16 operand: row-major, row stride ld (elements)
  const uint16_t* dense;
  int64_t ld;
  // the FP4 operand: K-major codes [rows][K/2] and scales (MXFP4 uint8 [rows][K/32], HiF4
  // uint32 [rows][K/64])
  const uint8_t* codes;
  const void* scales;
  float* Y;
  int64_t ldy;
};

typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

// 2^E as float32 for an E8M0 code (E = code - 127; 2^-127 is a float32 subnormal).
__device__ __forceinline__ float e8m0_f32(uint32_t code) {
  return code ? __uint_as_float(code << 23) : __uint_as_float(0x00400000u);
}

// Eight FP4 elements (one 32-bit word of codes, element 8w+i in nibble i) dequantized to bf16
// bits, exact, two per output word.  MXFP4: E2M1 magnitude times 2^E; HiF4: k (4+m)
// 2^(e-35-b) with b the level-2 + level-3 shift of each element's groups (elem0 = the first
// element's index inside its 64-block; pairs share their level-3 group).
template <int FMT>
__device__ __forceinline__ void dequant8(uint32_t w, int elem0, uint32_t scale, uint32_t out[4]) {
  if constexpr (FMT == 0) {
    const float sc = e8m0_f32(scale);
    out[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 0));
    out[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 1));
    out[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 2));
    out[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 3));
  } else {
    const uint32_t f = 4u + (scale & 3u);
    const int e = (int)((scale >> 2) & 63u) - 35;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int el = elem0 + 2 * i;  // both elements of the pair share level-2/3 groups
      const int sh = e - (int)((scale >> (8 + el / 8)) & 1u) - (int)((scale >> (16 + el / 4)) & 1u);
      const uint32_t c0 = (w >> (8 * i)) & 15u, c1 = (w >> (8 * i + 4)) & 15u;
      const uint32_t u0 = __float_as_uint(ldexpf((float)((c0 & 7u) * f), sh)) | ((c0 & 8u) << 28);
      const uint32_t u1 = __float_as_uint(ldexpf((float)((c1 & 7u) * f), sh)) | ((c1 & 8u) << 28);
      out[i] = (u0 >> 16) | (u1 & 0xFFFF0000u);  // exact: at most 6 significant bits
    }
  }
}

// Per-thread staging of one operand's K chunk.  Dense: R rows x 64 bf16 = 8 R 16-byte pieces,
// spread over the 256 threads.  FP4: R rows x 2 halves of 32 codes (16 bytes each).
template <int R>
struct DenseStage {
  static constexpr int kPieces = R * kChunk / 8;           // 16-byte pieces per chunk
  static constexpr int kPer = (kPieces + 255) / 256;       // per thread
  v4u v[kPer];
};
template <int R>
struct QuantStage {
  static constexpr int kPieces = 2 * R;                    // 16-byte code pieces per chunk
  static constexpr int kPer = (kPieces + 255) / 256;
  v4u c[kPer];
  uint32_t s[kPer];
};

template <int R>
__device__ __forceinline__ void load_dense(DenseStage<R>& st, const uint16_t* base, int64_t ld, int64_t row0,
                                           int64_t rows, int64_t k0, int64_t K, int tid) {
#pragma unroll
  for (int x = 0; x < DenseStage<R>::kPer; ++x) {
    const int piece = tid + 256 * x;
    const int r = piece / 8, seg = piece % 8;
    const int64_t row = row0 + r, k = k0 + 8 * seg;
    v4u z = {0u, 0u, 0u, 0u};
    if (piece < DenseStage<R>::kPieces && row < rows && k < K)
      z = *reinterpret_cast<const v4u*>(base + row * ld + k);
    st.v[x] = z;
  }
}

template <int R>
__device__ __forceinline__ void store_dense(const DenseStage<R>& st, uint16_t* lds, int tid) {
#pragma unroll
  for (int x = 0; x < DenseStage<R>::kPer; ++x) {
    const int piece = tid + 256 * x;
    if (piece < DenseStage<R>::kPieces) {
      const int r = piece / 8, seg = piece % 8;
      *reinterpret_cast<v4u*>(lds + r * kRowHalves + 8 * seg) = st.v[x];
    }
  }
}

template <int FMT, int R>
__device__ __forceinline__ void load_quant(QuantStage<R>& st, const uint8_t* codes, const void* scales,
                                           int64_t row0, int64_t rows, int64_t k0, int64_t K, int tid) {
#pragma unroll
  for (int x = 0; x < QuantStage<R>::kPer; ++x) {
    const int piece = tid + 256 * x;
    const int r = piece / 2, half = piece % 2;
    const int64_t row = row0 + r, k = k0 + 32 * half;
    v4u z = {0u, 0u, 0u, 0u};
    uint32_t s = 0u;
    if (piece < QuantStage<R>::kPieces && row < rows && k < K) {
      z = *reinterpret_cast<const v4u*>(codes + row * (K / 2) + k / 2);
      if constexpr (FMT == 0) s = reinterpret_cast<const uint8_t*>(scales)[row * (K / 32) + k / 32];
      else s = reinterpret_cast<const uint32_t*>(scales)[row * (K / 64) + k / 64];
    }
    st.c[x] = z;
    st.s[x] = s;
  }
}

template <int FMT, int R>
__device__ __forceinline__ void store_quant(const QuantStage<R>& st, uint16_t* lds, int tid) {
#pragma unroll
  for (int x = 0; x < QuantStage<R>::kPer; ++x) {
    const int piece = tid + 256 * x;
    if (piece < QuantStage<R>::kPieces) {
      const int r = piece / 2, half = piece % 2;
      uint16_t* dst = lds + r * kRowHalves + 32 * half;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        uint32_t o[4];
        // element index inside the HiF4 64-block: this half's 32 elements start at 32 half
        dequant8<FMT>(st.c[x][w], 32 * half + 8 * w, st.s[x], o);
        *reinterpret_cast<v4u*>(dst + 8 * w) = v4u{o[0], o[1], o[2], o[3]};
      }
    }
  }
}

// AQ: operand A (rows of Y) is the FP4 one (W16A4); otherwise operand B is (W4A16).  KG K
// groups of four waves share the output tile: group g takes chunks g, g + KG, ... with its own
// LDS buffers and register stages, and at the end groups 1.. park their accumulators in LDS
// and group 0 adds them in group order (deterministic) and stores the tile.
template <int FMT, bool AQ, int TM, int TN, int KG>
__global__ __launch_bounds__(256 * KG) void mixed_gemm_kernel(MixedParams p) {
  constexpr int BM = 64 * TM, BN = 64 * TN;
  constexpr int PER = TM * TN * 16 * 64;  // accumulator floats per wave
  union Smem {
    struct {
      uint16_t A[KG][2][BM * kRowHalves];
      uint16_t B[KG][2][BN * kRowHalves];
    } t;
    float red[KG > 1 ? (KG - 1) * 4 * PER : 1];
  };
  __shared__ __attribute__((aligned(16))) Smem sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = wave / 4, wl = wave % 4, tg = tid % 256;  // K group, wave and thread within it
  const int wm = wl % 2, wn = wl / 2;
  const int64_t row0 = (int64_t)blockIdx.y * BM, col0 = (int64_t)blockIdx.x * BN;
  const int64_t nchunks = (p.K + kChunk - 1) / kChunk;
  const int64_t nq = nchunks > g ? (nchunks - g + KG - 1) / KG : 0;  // this group's chunks
  const int64_t nrounds = (nchunks + KG - 1) / KG;                   // group 0's count
  uint16_t(*As)[BM * kRowHalves] = sm.t.A[g];
  uint16_t(*Bs)[BN * kRowHalves] = sm.t.B[g];

  using AStage = typename std::conditional<AQ, QuantStage<BM>, DenseStage<BM>>::type;
  using BStage = typename std::conditional<AQ, DenseStage<BN>, QuantStage<BN>>::type;
  AStage sa[2];
  BStage sb[2];
  auto load = [&](int64_t q, int r) {
    const int64_t k0 = (q * KG + g) * kChunk;
    if constexpr (AQ) {
      load_quant<FMT, BM>(sa[r], p.codes, p.scales, row0, p.M, k0, p.K, tg);
      load_dense<BN>(sb[r], p.dense, p.ld, col0, p.N, k0, p.K, tg);
    } else {
      load_dense<BM>(sa[r], p.dense, p.ld, row0, p.M, k0, p.K, tg);
      load_quant<FMT, BN>(sb[r], p.codes, p.scales, col0, p.N, k0, p.K, tg);
    }
  };
  auto store = [&](int r, int buf) {
    if constexpr (AQ) {
      store_quant<FMT, BM>(sa[r], As[buf], tg);
      store_dense<BN>(sb[r], Bs[buf], tg);
    } else {
      store_dense<BM>(sa[r], As[buf], tg);
      store_quant<FMT, BN>(sb[r], Bs[buf], tg);
    }
  };

  v16f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto compute = [&](int buf) {
#pragma unroll
    for (int kk = 0; kk < kChunk / 16; ++kk) {
      const int koff = 16 * kk + 8 * (lane / 32);
      v8bf a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = (wm * TM + i) * 32 + lane % 32;
        a[i] = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4u*>(As[buf] + r * kRowHalves + koff));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = (wn * TN + j) * 32 + lane % 32;
        b[j] = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4u*>(Bs[buf] + r * kRowHalves + koff));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };

  // The group's chunk q sits in register stage q % 2 from its load (two chunks ahead) until
  // its store into LDS buffer q % 2, one chunk ahead of its MFMAs.  Each round: issue chunk
  // q+2's loads, run chunk q's MFMAs, store chunk q+1 into the other buffer (last read during
  // chunk q-1, which the previous barrier closed), barrier.  Every group runs group 0's round
  // count (it has the most chunks), so all waves meet at every barrier.
  if (nq > 0) load(0, 0);
  if (nq > 1) load(1, 1);
  if (nq > 0) store(0, 0);
  __syncthreads();
  for (int64_t q0 = 0; q0 < nrounds; q0 += 2) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t q = q0 + u;
      if (q < nrounds) {
        if (q < nq) {
          if (q + 2 < nq) load(q + 2, u);
          compute(u);
          if (q + 1 < nq) store(1 - u, 1 - u);
        }
        __syncthreads();
      }
    }
  }

  if constexpr (KG > 1) {
    // every wave is past its last LDS read (the loop's final barrier): reuse LDS for the sums
    if (g > 0) {
      float* dst = sm.red + ((size_t)(g - 1) * 4 + wl) * PER;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) dst[((i * TN + j) * 16 + r) * 64 + lane] = acc[i][j][r];
    }
    __syncthreads();
    if (g > 0) return;
#pragma unroll
    for (int gg = 1; gg < KG; ++gg) {
      const float* src = sm.red + ((size_t)(gg - 1) * 4 + wl) * PER;
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
      const int64_t col = col0 + (wn * TN + j) * 32 + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = row0 + (wm * TM + i) * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (row < p.M && col < p.N) p.Y[row * p.ldy + col] = acc[i][j][r];
      }
    }
}

template <int FMT, bool AQ, int TM, int TN, int KG>
void launch_tile(const MixedParams& p, hipStream_t s) {
  const dim3 grid((unsigned)((p.N + 64 * TN - 1) / (64 * TN)), (unsigned)((p.M + 64 * TM - 1) / (64 * TM)));
  launch_timed(mixed_gemm_kernel<FMT, AQ, TM, TN, KG>, grid, dim3(256 * KG), 0u, s, p);
}

// Tile choice: the FP4 operand's dequantization is shared by the rows (W4A16) or columns
// (W16A4) of the tile, so the tile is as long as possible along the other operand while the
// grid still has at least 128 workgroups; the other side stays 64 wide.  Grids of 64 x 64
// tiles within the CUs that have at least 16 K chunks take four K groups per workgroup.
template <int FMT, bool AQ>
void launch_fmt(const MixedParams& p, hipStream_t s) {
  const int64_t along = AQ ? p.N : p.M, across = AQ ? p.M : p.N;
  auto wgs = [&](int64_t t) { return ((along + 64 * t - 1) / (64 * t)) * ((across + 63) / 64); };
  const int t = wgs(4) >= 128 ? 4 : wgs(2) >= 128 ? 2 : 1;
  const bool kgroups = t == 1 && wgs(1) <= 256 && (p.K + kChunk - 1) / kChunk >= 16;
  if constexpr (AQ) {
    if (t == 4) launch_tile<FMT, AQ, 1, 4, 1>(p, s);
    else if (t == 2) launch_tile<FMT, AQ, 1, 2, 1>(p, s);
    else if (kgroups) launch_tile<FMT, AQ, 1, 1, 4>(p, s);
    else launch_tile<FMT, AQ, 1, 1, 1>(p, s);
  } else {
    if (t == 4) launch_tile<FMT, AQ, 4, 1, 1>(p, s);
    else if (t == 2) launch_tile<FMT, AQ, 2, 1, 1>(p, s);
    else if (kgroups) launch_tile<FMT, AQ, 1, 1, 4>(p, s);
    else launch_tile<FMT, AQ, 1, 1, 1>(p, s);
  }
}

}  // namespace

void launch_mixed_gemm(int fmt, bool a_quantized, int64_t M, int64_t N, int64_t K, const uint16_t* dense,
                       int64_t ld, const uint8_t* codes, const void* scales, float* Y, int64_t ldy,
                       hipStream_t s) {
  if (M == 0 || N == 0) return;
  MixedParams p{M, N, K, dense, ld, codes, scales, Y, ldy};
  if (fmt == 0) {
    if (a_quantized) launch_fmt<0, true>(p, s);
    else launch_fmt<0, false>(p, s);
  } else {
    if (a_quantized) launch_fmt<1, true>(p, s);
    else launch_fmt<1, false>(p, s);
  }
}

}  // namespace resq
