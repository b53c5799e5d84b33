// Mixed-precision rollout GEMMs of the paper's precision ablation (Table 1): weight-only FP4
// (W4A16: Y = X Q(W)^T, bf16 activations) and activation-only FP4 (W16A4: Y = Q(X) W^T, bf16
// weights), float32 Y.
//
// Both run on gfx950's bf16 MFMA (v_mfma_f32_32x32x16_bf16, float32 accumulation).  Every
// FP4 value is exact in bf16 (an MXFP4 value has 2 significant bits, a HiF4 value
// k (4+m) 2^(e-35-b) at most 6), so an FP4 operand is dequantized to bf16 without rounding
// and every product is exact in float32; only the accumulation rounds.
//
// Operand roles.  The row operand A (rows of Y) is always bf16: X itself (W4A16), or Q(X)
// dequantized to bf16 by a row pass before the GEMM (W16A4: the activations are a few MB at
// rollout batch sizes, so writing them at 2 bytes per element costs nothing next to the bf16
// weights, and the GEMM then dequantizes nothing per output tile).  The column operand B is
// the weight: K-major FP4 codes + block scales (W4A16), dequantized in registers right before
// the MFMAs (MXFP4 by the scaled FP4 conversion, HiF4 by a per-block byte table), so HBM
// carries 4.25 (MXFP4) or 4.5 (HiF4) bits per weight; or bf16 rows (W16A4).
//
// Work split.  A workgroup owns a 32 TM x (32 TN WN) output tile: WN waves side by side along
// the columns, each owning 32 TM x 32 TN of it, all of them reading the same A rows.  KG such
// groups share the tile and split its K range in super-chunks of four rounds (super-chunk s
// goes to group s mod KG); at the end they add their accumulators through LDS in group order
// (deterministic).  Workgroups are
// dealt to the eight XCDs in contiguous ranges, row tiles fastest, so the workgroups that read
// one weight strip run on one XCD at about the same time and share its L2.
//
// Data movement.  K advances in rounds of 64.  Both operands go from global memory straight
// into LDS (buffer loads with the LDS destination, no register staging).  A copy instruction
// moves 64 lanes x 16 bytes; it is laid out to read whole 128-byte lines (8 rows x 128 bytes
// of A or bf16 B per round; for FP4 B, 8 columns x 128 bytes of codes, which span four
// rounds, so FP4 codes move in super-chunks of 256 K), since copies that touch many lines
// for few bytes each run far slower than the bytes alone would suggest.  In LDS each 128-byte
// row keeps its 16-byte segments XOR-swizzled by the row index and rows 8..15 of every 16
// swap neighbours, so the MFMA operand reads (16 bytes per lane, 32 rows) are free of bank
// conflicts.  A rows are copied once per group
// (each wave 4 TM / WN of the instructions) and read by all WN waves; B is private to its
// wave.  NS rounds are in flight; one barrier per round.  FP4 scales travel as one dword per
// lane, tile and round (MXFP4: the aligned dword holding the lane's scale byte).
//
// K order inside a round.  The sum over K may take any order, as long as A and B pair the
// same K.  Lane l (row or column l % 32, half h = l / 32) holds the 32 consecutive K elements
// 32 h .. 32 h + 31 of the round, and the MFMA of step kk (0..3) takes elements 8 kk .. 8 kk + 7
// of them: one 16-byte read per step for bf16, one 32-bit word of codes for FP4, whose
// 32-element span is exactly one MXFP4 block and one half of a HiF4 block.
//
// MFMA layouts (32x32x16 bf16): lane l holds row (A) / column (B) l % 32 and 8 K elements of
// the 16-wide step; accumulator register r of lane l is row 8 (r / 4) + 4 (l / 32) + r % 4,
// column l % 32.
#include <type_traits>

#include "kernels.h"
#include "device_fp4.h"
#include "quant_core.h"
#include "profiler.h"

namespace resq {
namespace {

typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr int kXcds = 8;
// Largest operand buffer a launch addresses (32-bit buffer offsets); kOut lies past every
// such buffer, so a copy from it reads zeros.
constexpr uint64_t kMaxBuffer = 0xFFFFFE00ull;
constexpr uint32_t kOut = 0xFFFFFF00u;

struct MixedParams {
  int64_t M, N, K;
  const void* a;        // bf16 rows, lda_b bytes apart
  uint32_t a_bytes, lda_b;
  const void* b;        // FP4 codes (K / 2 bytes per row) or bf16 rows, ldb_b bytes apart
  uint32_t b_bytes, ldb_b;
  const void* bs;       // FP4 scales: MXFP4 uint8 [N][K/32] (from byte bs_mis on), HiF4 uint32 [N][K/64]
  uint32_t bs_bytes, bs_mis;
  float* Y;
  int64_t ldy;
  uint32_t mt;          // row tiles
  uint32_t n_wg, per_xcd;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// 16 bytes per lane from buffer offset voff into LDS: lane l's bytes land at lds + 16 l.
__device__ __forceinline__ void copy16(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)lds, 16, voff, 0, 0, 0);
}

// 4 bytes per lane from buffer offset voff (4-byte aligned) into LDS: lane l's at lds + 4 l.
__device__ __forceinline__ void copy4(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)lds, 4, voff, 0, 0, 0);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt field is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Barrier that also waits for this wave's LDS reads but not for its LDS-destination copies
// (those are waited for with wait_vmcnt); the memory clobber keeps accesses on their side.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// 2^E as float32 for an E8M0 code (E = code - 127; 2^-127 is a float32 subnormal).
__device__ __forceinline__ float e8m0_f32(uint32_t code) {
  return code ? __uint_as_float(code << 23) : __uint_as_float(0x00400000u);
}

// Eight MXFP4 elements (one 32-bit word of codes, element i in nibble i) dequantized to bf16
// bits, exact, two per output word: E2M1 magnitude times 2^E through gfx950's scaled
// conversion (v_cvt_scalef32_pk_bf16_fp4).
__device__ __forceinline__ void mx_dequant8(uint32_t w, uint32_t scale, uint32_t out[4]) {
  const float sc = e8m0_f32(scale);
  out[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 0));
  out[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 1));
  out[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 2));
  out[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 3));
}

// HiF4 decoding by table (the lane's 32 elements of a round lie in one 64-block).  Per round:
// the bf16 patterns L[k] of k (4+m) 2^(e-35) for k = 0..7 (exact, L[0] = 0), split into
// their low and high bytes, four entries per dword, and the lane's level-2 (4) and level-3
// (8) shift bits.  Per 8 elements: the magnitudes k spread to bytes select the bytes of
// their entries (v_perm), the signs go into the high bytes of nonzero elements, the bytes
// pair up into bf16 values, and a saturating 16-bit subtraction of b << 7 lowers the
// exponent by the element's shift b (nonzero values keep biased exponents far above 2, and
// zero stays zero).
struct Hif4Table {
  uint32_t lo03, lo47, hi03, hi47;  // low / high bytes of L[0..3], L[4..7]
  uint32_t l2, l3;                  // level-2 bits of the lane's 4 groups of 8, level-3 of its 8 of 4
};

__device__ __forceinline__ Hif4Table hif4_table(uint32_t scale, int h) {
  const uint32_t f = 4u + (scale & 3u);
  const int e = (int)((scale >> 2) & 63u) - 35;
  uint32_t L[8];
  L[0] = 0u;
#pragma unroll
  for (int k = 1; k < 8; ++k) L[k] = __float_as_uint(ldexpf((float)(k * f), e)) >> 16;  // exact
  const uint32_t p01 = L[0] | (L[1] << 16), p23 = L[2] | (L[3] << 16);
  const uint32_t p45 = L[4] | (L[5] << 16), p67 = L[6] | (L[7] << 16);
  Hif4Table t;
  t.lo03 = __builtin_amdgcn_perm(p23, p01, 0x06040200u);
  t.hi03 = __builtin_amdgcn_perm(p23, p01, 0x07050301u);
  t.lo47 = __builtin_amdgcn_perm(p67, p45, 0x06040200u);
  t.hi47 = __builtin_amdgcn_perm(p67, p45, 0x07050301u);
  t.l2 = (scale >> (8 + 4 * h)) & 0xFu;
  t.l3 = (scale >> (16 + 8 * h)) & 0xFFu;
  return t;
}

typedef unsigned short v2u16 __attribute__((ext_vector_type(2)));

// Four elements: their nibbles in the low nibbles of the four bytes of sp; out0/out1 receive
// elements 0,1 / 2,3 as bf16 pairs, shifted down by b.
__device__ __forceinline__ void hif4_decode4(uint32_t sp, uint32_t b, const Hif4Table& t, uint32_t& out0,
                                             uint32_t& out1) {
  const uint32_t k = sp & 0x07070707u;
  const uint32_t lo = __builtin_amdgcn_perm(t.lo47, t.lo03, k);
  uint32_t hi = __builtin_amdgcn_perm(t.hi47, t.hi03, k);
  hi |= (sp << 4) & (k + 0x7F7F7F7Fu) & 0x80808080u;  // the sign bit of each nonzero element
  const v2u16 sub = __builtin_bit_cast(v2u16, b * 0x00800080u);
  out0 = __builtin_bit_cast(uint32_t, __builtin_elementwise_sub_sat(
                                          __builtin_bit_cast(v2u16, __builtin_amdgcn_perm(hi, lo, 0x05010400u)), sub));
  out1 = __builtin_bit_cast(uint32_t, __builtin_elementwise_sub_sat(
                                          __builtin_bit_cast(v2u16, __builtin_amdgcn_perm(hi, lo, 0x07030602u)), sub));
}

// Eight elements of step kk (elements 8 kk .. 8 kk + 7 of the lane's 32): one level-2 group,
// two level-3 groups.
template <int KK>
__device__ __forceinline__ void hif4_decode8(uint32_t w, const Hif4Table& t, uint32_t out[4]) {
  const uint32_t b2 = (t.l2 >> KK) & 1u;
  const uint32_t ba = b2 + ((t.l3 >> (2 * KK)) & 1u), bb = b2 + ((t.l3 >> (2 * KK + 1)) & 1u);
  const uint32_t ta = __builtin_amdgcn_perm(w, w, 0x0C010C00u), tb = __builtin_amdgcn_perm(w, w, 0x0C030C02u);
  hif4_decode4(ta | (ta << 4), ba, t, out[0], out[1]);
  hif4_decode4(tb | (tb << 4), bb, t, out[2], out[3]);
}

template <bool BQ, int TM, int TN, int WN, int KG, int NS>
struct MixGeo {
  static constexpr int AI = 4 * TM;                    // A copies (1 KB, 8 rows) per round
  static constexpr int APW = AI / WN;                  // of which each wave issues
  static constexpr int BR = BQ ? 0 : 4 * TN;           // bf16 B copies per wave and round
  static constexpr int SC = BQ ? TN * 256 : 0;         // FP4 scale bytes per wave and round
  static constexpr int RSLOT = AI * 1024 + WN * (BR * 1024 + SC);  // round slot
  static constexpr int RB = BQ ? 2 : 0;                // super-chunk slots
  static constexpr int BSLOT = BQ ? WN * 4 * TN * 1024 : 0;        // super-chunk slot
  static constexpr int GROUP = NS * RSLOT + RB * BSLOT;
  static constexpr int RED = (KG - 1) * WN * TM * TN * 16 * 64 * 4;
  static constexpr int LDS = KG * GROUP > RED ? KG * GROUP : RED;
  // copies issued in a round of phase q (round index mod 4)
  static constexpr int jw(int q) { return APW + BR + (BQ ? TN : 0) + (BQ && q == 0 ? 4 * TN : 0); }
  // copies the wait at a round of phase q leaves in flight: those of the NS - 2 later rounds
  static constexpr int inflight(int q) {
    int n = 0;
    for (int u = 1; u <= NS - 2; ++u) n += jw((q + u) % 4);
    return n;
  }
  static constexpr bool ok = AI % WN == 0 && WN % 2 == 0 && (NS == 2 || NS == 4) &&
                             inflight(0) + jw(0) < 64 && inflight(1) + jw(1) < 64 &&
                             inflight(2) + jw(2) < 64 && inflight(3) + jw(3) < 64 &&
                             LDS <= 160 * 1024;
};

// A and bf16 B rows in LDS: row r (128 bytes of one 64-K round) at position
// r ^ ((r / 8) % 2) (rows 8..15 of every 16 swap neighbours), its 16-byte segment s at slot
// s ^ (r % 8).  The MFMA operand reads of 16 consecutive rows (one segment each) then fall
// in 16 different 16-byte bank groups of the 256 bytes the two row parities cover.  A copy
// instruction moves the 8 rows of 8 consecutive positions: lane l fills slot l % 8 of
// position l / 8 with the segment that belongs there.  FP4 codes: column c's 128 bytes of one
// super-chunk (256 K: segment s = round s / 2, lane half s % 2) the same way.
__device__ __forceinline__ uint32_t swz(int row, int seg) {
  return (uint32_t)((row ^ ((row >> 3) & 1)) * 128 + 16 * (seg ^ (row & 7)));
}

template <int FMT, bool BQ, int TM, int TN, int WN, int KG, int NS>
__global__ __launch_bounds__(64 * WN * KG) void mixed_gemm_kernel(MixedParams p) {
  using G = MixGeo<BQ, TM, TN, WN, KG, NS>;
  static_assert(G::ok, "configuration out of range");
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  const uint32_t bid = blockIdx.x;
  const uint32_t wg = (bid % kXcds) * p.per_xcd + bid / kXcds;
  if (wg >= p.n_wg) return;
  const uint32_t tm = wg % p.mt, tn = wg / p.mt;
  const int lane = threadIdx.x & 63, h = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = wave / WN, wn = wave % WN;
  const int64_t row0 = (int64_t)tm * 32 * TM;
  const int64_t colw = ((int64_t)tn * WN + wn) * 32 * TN;  // this wave's first column
  const uint32_t nchunks = (uint32_t)((p.K + 63) / 64);
  const uint32_t nsuper = (nchunks + 3) / 4;
  const uint32_t nrounds = 4 * ((nsuper + KG - 1) / KG);  // per group, a multiple of 4
  uint8_t* rring = smem + (size_t)g * G::GROUP;
  uint8_t* bring = rring + NS * G::RSLOT;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.a, p.a_bytes), rb = make_rsrc(p.b, p.b_bytes);
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(p.bs, p.bs_bytes);
  // the copy lane's row within the 8 rows of an instruction x (x % 2 = par) and the global
  // segment it moves
  auto crow = [&](int par) { return (lane >> 3) ^ par; };
  auto cseg = [&](int par) { return (lane & 7) ^ crow(par); };
  const int apar = wn & 1;  // WN is even: every A instruction of this wave, x = wn + WN y

  // Round-0 offsets of this lane's copies, and kOut masks for rows / columns outside the
  // matrix: an offset OR-ed with kOut lies past every buffer, so its copy reads zeros.
  uint32_t aoff[G::APW], amask[G::APW];
#pragma unroll
  for (int y = 0; y < G::APW; ++y) {
    const int64_t row = row0 + 8 * (wn + WN * y) + crow(apar);
    aoff[y] = row < p.M ? (uint32_t)row * p.lda_b + 16u * cseg(apar) : 0u;
    amask[y] = row < p.M ? 0u : kOut;
  }
  // B copies: bf16 rows per round (BR) or FP4 super-chunks (4 TN), 8 columns each
  constexpr int BX = BQ ? 4 * TN : G::BR;
  uint32_t boff[BX], bmask[BX];
#pragma unroll
  for (int x = 0; x < BX; ++x) {
    const int64_t col = colw + 8 * x + crow(x & 1);
    boff[x] = col < p.N ? (uint32_t)col * p.ldb_b + 16u * cseg(x & 1) : 0u;
    bmask[x] = col < p.N ? 0u : kOut;
  }
  uint32_t soff[TN], smask[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int64_t col = colw + 32 * j + l32;
    smask[j] = col < p.N ? 0u : kOut;
    if constexpr (BQ) {
      if constexpr (FMT == 0) soff[j] = col < p.N ? (uint32_t)(col * (p.K / 32)) + h + p.bs_mis : 0u;
      else soff[j] = col < p.N ? (uint32_t)(col * (p.K / 64)) * 4u : 0u;
    }
  }

  // Round t of this group is chunk 4 (g + KG (t / 4)) + t % 4: each group takes whole
  // super-chunks, so the FP4 codes of a column are read 128 contiguous bytes at a time.
  auto chunk_of = [&](uint32_t t) { return 4u * (g + KG * (t >> 2)) + (t & 3u); };
  auto super_copies = [&](uint32_t S) {  // FP4 super-chunk S of this group into its slot
    const uint32_t k4 = g + KG * S;
    uint8_t* dst = bring + (S % G::RB) * G::BSLOT + wn * 4 * TN * 1024;
    const uint32_t kout0 = 256ull * k4 + 32u * cseg(0) < (uint64_t)p.K ? 0u : kOut;
    const uint32_t kout1 = 256ull * k4 + 32u * cseg(1) < (uint64_t)p.K ? 0u : kOut;
#pragma unroll
    for (int x = 0; x < BX; ++x) copy16(rb, dst + x * 1024, (boff[x] + 128u * k4) | bmask[x] | (x & 1 ? kout1 : kout0));
  };
  // Issue slot u: round u's A rows, scales or bf16 B rows into round slot u % NS (= rs_),
  // and, at every fourth slot, FP4 super-chunk u / 4.
  auto issue = [&](uint32_t u, int rs_, bool super) {
    const uint32_t c = chunk_of(u);
    // kOut where the 8 K elements a copy lane moves lie past K
    const uint32_t kout = 64ull * c + 8u * cseg(apar) < (uint64_t)p.K ? 0u : kOut;
    const uint32_t kout0 = 64ull * c + 8u * cseg(0) < (uint64_t)p.K ? 0u : kOut;
    const uint32_t kout1 = 64ull * c + 8u * cseg(1) < (uint64_t)p.K ? 0u : kOut;
    uint8_t* st = rring + rs_ * G::RSLOT;
#pragma unroll
    for (int y = 0; y < G::APW; ++y) copy16(ra, st + (wn + WN * y) * 1024, (aoff[y] + 128u * c) | amask[y] | kout);
    uint8_t* sw = st + G::AI * 1024 + wn * (G::BR * 1024 + G::SC);
    if constexpr (BQ) {
      const uint32_t skout = 64ull * c + 32u * h < (uint64_t)p.K ? 0u : kOut;  // this lane's block
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const uint32_t so = FMT == 0 ? (soff[j] + 2u * c) & ~3u : soff[j] + 4u * c;
        copy4(rs, sw + j * 256, so | smask[j] | skout);
      }
      if (super) super_copies(u >> 2);
    } else {
#pragma unroll
      for (int x = 0; x < BX; ++x) copy16(rb, sw + x * 1024, (boff[x] + 128u * c) | bmask[x] | (x & 1 ? kout1 : kout0));
    }
  };

  v16f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto compute = [&](uint32_t t, int rs_) {
    const uint8_t* st = rring + rs_ * G::RSLOT;
    const uint8_t* sw = st + G::AI * 1024 + wn * (G::BR * 1024 + G::SC);
    v4u bc[TN];
    uint32_t sc[TN];
    [[maybe_unused]] Hif4Table tab[TN];
    if constexpr (BQ) {
      const uint8_t* bs = bring + ((t >> 2) % G::RB) * G::BSLOT + wn * 4 * TN * 1024;
      const uint32_t c = chunk_of(t);
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        bc[j] = *reinterpret_cast<const v4u*>(bs + swz(32 * j + l32, 2 * (int)(t & 3u) + h));
        sc[j] = *reinterpret_cast<const uint32_t*>(sw + j * 256 + 4 * lane);
        if constexpr (FMT == 0) sc[j] = (sc[j] >> (8 * ((soff[j] + 2u * c) & 3u))) & 0xFFu;
        else tab[j] = hif4_table(sc[j], h);
      }
    }
    // every LDS read of the round first, so the MFMAs of the four steps issue back to back
    v4u a[4][TM], bd[4][BQ ? 1 : TN];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int i = 0; i < TM; ++i) a[kk][i] = *reinterpret_cast<const v4u*>(st + swz(32 * i + l32, 4 * h + kk));
    if constexpr (!BQ) {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int j = 0; j < TN; ++j) bd[kk][j] = *reinterpret_cast<const v4u*>(sw + swz(32 * j + l32, 4 * h + kk));
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the reads ahead of the MFMAs
    auto step = [&](auto kc) {
      constexpr int kk = decltype(kc)::value;
      v8bf b[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        if constexpr (BQ) {
          uint32_t o[4];
          if constexpr (FMT == 0) mx_dequant8(bc[j][kk], sc[j], o);
          else hif4_decode8<kk>(bc[j][kk], tab[j], o);
          b[j] = __builtin_bit_cast(v8bf, v4u{o[0], o[1], o[2], o[3]});
        } else {
          b[j] = __builtin_bit_cast(v8bf, bd[kk][j]);
        }
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, a[kk][i]), b[j], acc[i][j], 0, 0, 0);
    };
    step(std::integral_constant<int, 0>{});
    step(std::integral_constant<int, 1>{});
    step(std::integral_constant<int, 2>{});
    step(std::integral_constant<int, 3>{});
  };

  // Round t: wait until this wave's copies of issue slots <= t have landed (those of the
  // NS - 2 later slots stay in flight), a barrier (every wave's copies of round t have landed
  // and every wave has finished reading round t - 1, whose round slot and, after the last
  // round of a super-chunk, super-chunk slot are refilled next), issue slot t + NS - 1, then
  // round t's MFMAs.  FP4 super-chunk S is issued with round 4 S, so it has landed by round
  // 4 S; its slot (S mod 2) was last read in rounds 4 S - 8 .. 4 S - 5, before the barrier of
  // round 4 S - NS + 1 that precedes its copies (NS <= 4).  The loop is unrolled four times,
  // so the round slots (NS divides 4) and the wait counts are compile-time.
#pragma unroll
  for (int u = 0; u < NS - 1; ++u) issue(u, u, u % 4 == 0);
  for (uint32_t t0 = 0; t0 < nrounds; t0 += 4) {
    auto round = [&](auto qc) {
      constexpr int q = decltype(qc)::value;
      wait_vmcnt<G::inflight(q)>();
      lds_barrier();
      issue(t0 + q + NS - 1, (q + NS - 1) % NS, (q + NS - 1) % 4 == 0);
      compute(t0 + q, q % NS);
    };
    round(std::integral_constant<int, 0>{});
    round(std::integral_constant<int, 1>{});
    round(std::integral_constant<int, 2>{});
    round(std::integral_constant<int, 3>{});
  }
  wait_vmcnt<0>();  // the copies of the slots past the end have landed before LDS is reused

  if constexpr (KG > 1) {
    constexpr int PER = TM * TN * 16 * 64;  // accumulator floats per wave
    float* red = reinterpret_cast<float*>(smem);
    lds_barrier();
    if (g > 0) {
      float* dst = red + ((size_t)(g - 1) * WN + wn) * PER;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) dst[((i * TN + j) * 16 + r) * 64 + lane] = acc[i][j][r];
    }
    lds_barrier();
    if (g > 0) return;
#pragma unroll
    for (int gg = 1; gg < KG; ++gg) {
      const float* src = red + ((size_t)(gg - 1) * WN + wn) * PER;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] += src[((i * TN + j) * 16 + r) * 64 + lane];
    }
  }

#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int64_t col = colw + 32 * j + l32;
      if (col >= p.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = row0 + 32 * i + 8 * (r >> 2) + 4 * h + (r & 3);
        if (row < p.M) p.Y[row * p.ldy + col] = acc[i][j][r];
      }
    }
}

// Q(X) along rows, written as the dequantized values in bf16 (exact): one lane per 4
// elements, grid (ceil(cols / 1024), rows).  out is 8-byte aligned with ldo % 4 == 0.
template <int FMT, bool VEC>
__global__ __launch_bounds__(256) void quant_rows_bf16_kernel(const uint16_t* __restrict__ x, int64_t rows,
                                                              int64_t cols, int64_t ld,
                                                              uint16_t* __restrict__ out, int64_t ldo) {
  const int64_t j4 = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (4 * j4 >= cols) return;  // whole blocks drop out together (cols % block == 0)
  for (int64_t row = blockIdx.y; row < rows; row += gridDim.y) {
    float v[4];
    const int64_t i = row * ld + 4 * j4;
    if constexpr (VEC) {
      const uint2 t = *reinterpret_cast<const uint2*>(x + i);
      v[0] = bf16_to_f32(t.x & 0xFFFFu); v[1] = bf16_to_f32(t.x >> 16);
      v[2] = bf16_to_f32(t.y & 0xFFFFu); v[3] = bf16_to_f32(t.y >> 16);
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] = bf16_to_f32(x[i + k]);
    }
    const Quad q = quantize_quad<FMT>(v);
    // the values carry at most 6 significant bits: their float32 patterns end in 16 zero bits
    const uint32_t lo = (__float_as_uint(q.val[0]) >> 16) | (__float_as_uint(q.val[1]) & 0xFFFF0000u);
    const uint32_t hi = (__float_as_uint(q.val[2]) >> 16) | (__float_as_uint(q.val[3]) & 0xFFFF0000u);
    *reinterpret_cast<uint2*>(out + row * ldo + 4 * j4) = make_uint2(lo, hi);
  }
}

// Tile configurations (TM, TN, WN, KG, NS), instantiated for both operand kinds where they
// fit (MixGeo::ok).
struct MixPlan {
  int tm, tn, wn, kg, ns;
};
#define RESQ_MIXED_CONFIGS(X) \
  X(2, 1, 4, 1, 4) X(1, 1, 4, 1, 4) X(8, 1, 4, 1, 2) X(1, 1, 2, 4, 4) X(1, 1, 4, 2, 4) X(2, 1, 2, 4, 2) \
  X(1, 1, 2, 2, 4) X(2, 2, 4, 1, 2) X(1, 2, 4, 1, 2)

template <int FMT, bool BQ, int TM, int TN, int WN, int KG, int NS>
void launch_cfg(MixedParams p, hipStream_t s) {
  using G = MixGeo<BQ, TM, TN, WN, KG, NS>;
  if constexpr (G::ok) {
    p.mt = (uint32_t)((p.M + 32 * TM - 1) / (32 * TM));
    const uint64_t nt = (uint64_t)((p.N + 32 * TN * WN - 1) / (32 * TN * WN));
    p.n_wg = (uint32_t)(p.mt * nt);
    p.per_xcd = (p.n_wg + kXcds - 1) / kXcds;
    launch_timed(mixed_gemm_kernel<FMT, BQ, TM, TN, WN, KG, NS>, dim3(p.per_xcd * kXcds), dim3(64 * WN * KG),
                 (uint32_t)G::LDS, s, p);
  }
}

template <bool BQ>
bool plan_fits(const MixPlan& c) {
#define RESQ_MX_FIT(TM, TN, WN, KG, NS) \
  if (c.tm == TM && c.tn == TN && c.wn == WN && c.kg == KG && c.ns == NS) return MixGeo<BQ, TM, TN, WN, KG, NS>::ok;
  RESQ_MIXED_CONFIGS(RESQ_MX_FIT)
#undef RESQ_MX_FIT
  return false;
}

template <int FMT, bool BQ>
void launch_plan(const MixPlan& c, const MixedParams& p, hipStream_t s) {
#define RESQ_MX_CASE(TM, TN, WN, KG, NS) \
  if (c.tm == TM && c.tn == TN && c.wn == WN && c.kg == KG && c.ns == NS) return launch_cfg<FMT, BQ, TM, TN, WN, KG, NS>(p, s);
  RESQ_MIXED_CONFIGS(RESQ_MX_CASE)
#undef RESQ_MX_CASE
}

// Plan choice (measured on MI355X at the m = 256 decode shapes).  Wide grids (many column
// tiles): 64 x 128 tiles, one per four waves; HiF4 weights take 256-row tiles instead, so
// each dequantized weight fragment feeds eight MFMAs (its dequantization costs some 40 VALU
// instructions per 8 elements).  Long K with few columns: 32 x 64 tiles in K groups.
// Otherwise 32-row tiles in two K groups, 64 columns wide if that still fits the 256 CUs in
// one round of workgroups, else 128 (HiF4: 64 x 64 in four K groups).  bf16 weights (W16A4):
// 64 x 256, 32 x 64 in two K groups, or the same small tiles.
static_assert(MixGeo<true, 2, 1, 4, 1, 4>::ok && MixGeo<true, 1, 1, 4, 1, 4>::ok && MixGeo<true, 8, 1, 4, 1, 2>::ok &&
                  MixGeo<true, 1, 1, 2, 4, 4>::ok && MixGeo<true, 2, 1, 2, 4, 2>::ok && MixGeo<true, 1, 1, 4, 2, 4>::ok &&
                  MixGeo<true, 1, 1, 2, 2, 4>::ok && MixGeo<false, 2, 2, 4, 1, 2>::ok && MixGeo<false, 1, 2, 4, 1, 2>::ok &&
                  MixGeo<false, 1, 1, 2, 2, 4>::ok && MixGeo<false, 1, 1, 4, 2, 4>::ok,
              "every plan choose() returns fits");
template <int FMT, bool BQ>
MixPlan choose(int64_t M, int64_t N, int64_t K) {
  const bool small = M <= 32;
  const int64_t mt64 = (M + 63) / 64, nchunks = (K + 63) / 64;
  const bool one_round = ((M + 31) / 32) * ((N + 63) / 64) <= 256;  // 32 x 64 tiles fit the CUs
  const MixPlan narrow = one_round ? MixPlan{1, 1, 2, 2, 4} : MixPlan{1, 1, 4, 2, 4};
  MixPlan c{};
  if constexpr (BQ) {
    if (mt64 * ((N + 127) / 128) >= 512)
      c = FMT == 1 && M >= 192 ? MixPlan{8, 1, 4, 1, 2} : MixPlan{small ? 1 : 2, 1, 4, 1, 4};
    else if (nchunks >= 64)
      c = MixPlan{1, 1, 2, 4, 4};
    else
      c = FMT == 1 && !small ? MixPlan{2, 1, 2, 4, 2} : narrow;
  } else {
    if (mt64 * ((N + 255) / 256) >= 256)
      c = MixPlan{small ? 1 : 2, 2, 4, 1, 2};
    else if (nchunks >= 64)
      c = MixPlan{1, 1, 2, 2, 4};
    else
      c = narrow;
  }
  return c;
}

// Rows of A (B) per launch so that every operand buffer of a launch stays within kMaxBuffer
// bytes (mixed_gemm_supported guarantees at least one row fits).
inline int64_t piece(int64_t row_bytes, int64_t last_bytes, int64_t per_row_extra) {
  int64_t n = (int64_t)(kMaxBuffer - last_bytes) / row_bytes + 1;
  if (per_row_extra > 0) n = std::min<int64_t>(n, (int64_t)kMaxBuffer / per_row_extra);
  return n > 256 ? n / 256 * 256 : n;
}

template <int FMT, bool BQ>
void launch_op(int64_t M, int64_t N, int64_t K, const uint16_t* a, int64_t lda, const void* b, int64_t ldb_b,
               const void* bs, float* Y, int64_t ldy, hipStream_t s) {
  const MixPlan c = choose<FMT, BQ>(M, N, K);
  const int64_t a_row = lda * 2, b_last = BQ ? K / 2 : K * 2;
  const int64_t bs_row = BQ ? (FMT == 0 ? K / 32 : K / 16) : 0;
  const int64_t mstep = piece(a_row, K * 2, 0), nstep = piece(ldb_b, b_last, bs_row);
  for (int64_t m0 = 0; m0 < M; m0 += mstep) {
    const int64_t mp = std::min(mstep, M - m0);
    for (int64_t n0 = 0; n0 < N; n0 += nstep) {
      const int64_t np = std::min(nstep, N - n0);
      MixedParams p{};
      p.M = mp;
      p.N = np;
      p.K = K;
      p.a = a + m0 * lda;
      p.a_bytes = (uint32_t)((mp - 1) * a_row + K * 2);
      p.lda_b = (uint32_t)a_row;
      p.b = reinterpret_cast<const uint8_t*>(b) + n0 * ldb_b;
      p.b_bytes = (uint32_t)((np - 1) * ldb_b + b_last);
      p.ldb_b = (uint32_t)ldb_b;
      // MXFP4 scales are read as the aligned dwords around them (base rounded down to 4
      // bytes); an aligned dword never crosses a page, so the bytes around the scales that
      // these dwords take along are readable
      const uintptr_t sp = BQ ? reinterpret_cast<uintptr_t>(bs) + (uintptr_t)(n0 * bs_row) : 0u;
      p.bs = reinterpret_cast<const void*>(sp & ~(uintptr_t)3);
      p.bs_mis = (uint32_t)(sp & 3u);
      p.bs_bytes = (uint32_t)((p.bs_mis + np * bs_row + 3) / 4 * 4);
      p.Y = Y + m0 * ldy + n0;
      p.ldy = ldy;
      launch_plan<FMT, BQ>(c, p, s);
    }
  }
}

}  // namespace

bool mixed_gemm_supported(int64_t K, int64_t lda, int64_t ldb, bool b_quantized) {
  const int64_t b_row = b_quantized ? K / 2 : 2 * ldb;
  return 2 * K <= (int64_t)kMaxBuffer / 2 && 2 * lda <= (int64_t)kMaxBuffer / 2 && b_row <= (int64_t)kMaxBuffer / 2;
}

void launch_quant_rows_bf16(int fmt, const uint16_t* x, int64_t rows, int64_t cols, int64_t ld, uint16_t* out,
                            int64_t ldo, hipStream_t s) {
  if (rows == 0 || cols == 0) return;
  const dim3 grid((unsigned)((cols / 4 + 255) / 256), (unsigned)(rows < 65535 ? rows : 65535));
  const bool vec = (uintptr_t)x % 8 == 0 && ld % 4 == 0;
#define RESQ_QRB(F, V) hipLaunchKernelGGL((quant_rows_bf16_kernel<F, V>), grid, dim3(256), 0, s, x, rows, cols, ld, out, ldo)
  if (fmt == 0) { if (vec) RESQ_QRB(0, true); else RESQ_QRB(0, false); }
  else { if (vec) RESQ_QRB(1, true); else RESQ_QRB(1, false); }
#undef RESQ_QRB
}

void launch_mixed_gemm(int fmt, int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                       const uint8_t* b_codes, const void* b_scales, const uint16_t* b_dense, int64_t ldb,
                       float* Y, int64_t ldy, hipStream_t s) {
  if (M == 0 || N == 0) return;
  if (b_codes == nullptr) launch_op<0, false>(M, N, K, A, lda, b_dense, ldb * 2, nullptr, Y, ldy, s);
  else if (fmt == 0) launch_op<0, true>(M, N, K, A, lda, b_codes, K / 2, b_scales, Y, ldy, s);
  else launch_op<1, true>(M, N, K, A, lda, b_codes, K / 2, b_scales, Y, ldy, s);
}

}  // namespace resq
