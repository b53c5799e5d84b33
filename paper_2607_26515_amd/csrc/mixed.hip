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
// bf16 rows or of FP4 codes), the workgroup writes them to LDS as bf16 rows (K contiguous,
// rows padded by 16 bytes), and each wave runs TM x TN x 4 MFMAs (K = 16 each) from LDS.  The
// next chunk's global loads are issued before the current chunk's MFMAs.
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

// Eight FP4 elements (one 32-bit word of codes, element 8w+i in nibble i) dequantized to bf16
// bits, exact.  MXFP4: magnitude in {0, .5, 1, 1.5, 2, 3, 4, 6} times 2^E; HiF4: k (4+m)
// 2^(e-35-b) with b the level-2 + level-3 shift of each element's groups.
template <int FMT>
__device__ __forceinline__ void dequant8(uint32_t w, int elem0, uint32_t scale, uint32_t out[4]) {
  uint32_t h[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t c = (w >> (4 * i)) & 15u;
    float v;
    if constexpr (FMT == 0) {
      v = ldexpf(e2m1_mag(c & 7u), (int)scale - 127);
    } else {
      const int e = (int)(scale & 0xFFu) >> 2, m = (int)(scale & 3u);
      const int el = elem0 + i;  // element index inside the 64-block
      const int b = (int)((scale >> (8 + el / 8)) & 1u) + (int)((scale >> (16 + el / 4)) & 1u);
      v = ldexpf((float)((c & 7u) * (uint32_t)(4 + m)), e - 35 - b);
    }
    const uint32_t u = __float_as_uint(v) | ((c & 8u) << 28);  // the code's sign, -0 kept
    h[i] = u >> 16;  // exact: at most 6 significant bits
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = h[2 * i] | (h[2 * i + 1] << 16);
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

// AQ: operand A (rows of Y) is the FP4 one (W16A4); otherwise operand B is (W4A16).
template <int FMT, bool AQ, int TM, int TN>
__global__ __launch_bounds__(256) void mixed_gemm_kernel(MixedParams p) {
  constexpr int BM = 64 * TM, BN = 64 * TN;
  __shared__ __attribute__((aligned(16))) uint16_t As[BM * kRowHalves];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * kRowHalves];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % 2, wn = wave / 2;
  const int64_t row0 = (int64_t)blockIdx.y * BM, col0 = (int64_t)blockIdx.x * BN;
  const int64_t nchunks = (p.K + kChunk - 1) / kChunk;

  using AStage = typename std::conditional<AQ, QuantStage<BM>, DenseStage<BM>>::type;
  using BStage = typename std::conditional<AQ, DenseStage<BN>, QuantStage<BN>>::type;
  AStage sa;
  BStage sb;
  auto load = [&](int64_t c) {
    const int64_t k0 = c * kChunk;
    if constexpr (AQ) {
      load_quant<FMT, BM>(sa, p.codes, p.scales, row0, p.M, k0, p.K, tid);
      load_dense<BN>(sb, p.dense, p.ld, col0, p.N, k0, p.K, tid);
    } else {
      load_dense<BM>(sa, p.dense, p.ld, row0, p.M, k0, p.K, tid);
      load_quant<FMT, BN>(sb, p.codes, p.scales, col0, p.N, k0, p.K, tid);
    }
  };

  v16f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  load(0);
  for (int64_t c = 0; c < nchunks; ++c) {
    if constexpr (AQ) {
      store_quant<FMT, BM>(sa, As, tid);
      store_dense<BN>(sb, Bs, tid);
    } else {
      store_dense<BM>(sa, As, tid);
      store_quant<FMT, BN>(sb, Bs, tid);
    }
    __syncthreads();
    if (c + 1 < nchunks) load(c + 1);  // in flight during this chunk's MFMAs
#pragma unroll
    for (int kk = 0; kk < kChunk / 16; ++kk) {
      const int koff = 16 * kk + 8 * (lane / 32);
      v8bf a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = (wm * TM + i) * 32 + lane % 32;
        a[i] = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4u*>(As + r * kRowHalves + koff));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = (wn * TN + j) * 32 + lane % 32;
        b[j] = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4u*>(Bs + r * kRowHalves + koff));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();  // every wave is done reading this chunk before the next one is stored
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

template <int FMT, bool AQ>
void launch_fmt(const MixedParams& p, hipStream_t s) {
  // 128 x 128 tiles when they give at least one workgroup per CU, else 64 x 64
  const int64_t big = ((p.M + 127) / 128) * ((p.N + 127) / 128);
  if (big >= 256) {
    const dim3 grid((unsigned)((p.N + 127) / 128), (unsigned)((p.M + 127) / 128));
    launch_timed(mixed_gemm_kernel<FMT, AQ, 2, 2>, grid, dim3(256), 0u, s, p);
  } else {
    const dim3 grid((unsigned)((p.N + 63) / 64), (unsigned)((p.M + 63) / 64));
    launch_timed(mixed_gemm_kernel<FMT, AQ, 1, 1>, grid, dim3(256), 0u, s, p);
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
