// FP4 GEMM on gfx950 scaled MFMA (v_mfma_scale_f32_32x32x64_f8f6f4):
//     Y[M][N] = Q(X) Q(W)^T  (+ S(Q(dX)) Q(W)^T into the same accumulators)   (Eq. 1, Eq. 4)
//
// MFMA operand layout (32x32x64): lane l holds row (A) / column (B) l%32 and the 32
// consecutive K elements (l/32)*32 .. +31 of the 64-wide K step, packed 4 bits (FP4) or 6
// bits (FP6) per element from bit 0 upwards; its E8M0 scale covers those 32 elements.
// Accumulator register r of lane l is row 8*(r/4) + 4*(l/32) + r%4, column l%32.
// Operands arrive "fragment-major" (pack.hip): fragment (tile, kb) is 64 consecutive lane
// records, plus one scale byte per lane in a separate array; all arrays of operand A (every
// term) share one buffer, and so do those of operand B.
//
// MXFP4 maps directly: E2M1 codes and E8M0 scales are the MFMA's own formats.
// HiF4: the level-1 scale s1 = 2^e (1 + m/4) is not a power of two, so no FP4/FP6 operand
// can carry it.  The activation value V 2^(e-37) (V <= 196) is split into two exact E2M3
// operands (hi, lo) and the weight element k 2^-b is an exact BF6 E3M2 operand with E8M0
// 2^(e_w - 35); the remaining weight factor (4 + m_w) is constant per output column, i.e. per
// lane, and is applied once per 64-K step: acc += (4 + m_w) * P_step.  Each tile's fold is
// issued after the next tile's MFMAs, so it runs under MFMA execution.
//
// Data movement.  A workgroup of WM x WN waves owns a (WM*TM*32) x (WN*TN*32) output tile.
// Each K step's operand bytes (A fragments of every term, B fragments, their scale bytes)
// are copied from global memory straight into an LDS stage by buffer loads with an LDS
// destination (no registers in between).  Every wave issues the same fixed number of 16-,
// 12- and 4-byte copy instructions per stage, so one explicit vmcnt wait per step tells a
// wave that its share of the next stage has landed, and one barrier publishes the stage to
// the other waves.  NS stages are in flight; the waves read their MFMA operands for step
// k+1 from LDS while the MFMAs of step k run.  The buffer descriptors and each lane's
// offsets are fixed for the whole loop (the K advance is the instruction's scalar offset);
// lanes of tiles past the edge copy zeros, and K steps past the end are copied through a
// zero-size buffer, so the loop has no data branches.
//
// K groups.  A workgroup may hold KG groups of WM x WN waves that share the output tile and
// split each stage's K range: a stage carries KG consecutive K steps and group g multiplies
// step g of it, so each barrier is amortised over KG steps and every SIMD holds KG waves
// with independent MFMA chains.  At the end the groups' accumulators are summed through LDS
// in group order (deterministic).  Decode-sized grids, which cannot fill the SIMDs with
// output tiles, use this.
//
// Workgroups are mapped to tiles in contiguous chunks per XCD (workgroup b runs on XCD
// b % 8), so tiles that share a weight column block run on the same XCD and share its L2.
// With a K split the split index varies slowest: an XCD's chunk then covers one K range of
// a block of tiles, whose A rows and B columns over that range it reads once, instead of
// every K range of fewer tiles (the ranges share no operand bytes).
#include "kernels.h"
#include "device_fp4.h"
#include "gemm_geo.h"
#include "profiler.h"


namespace resq {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v3i __attribute__((ext_vector_type(3)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr int kXcds = 8;

struct GemmParams {
  int64_t M, N, K, nkb, mt_tiles, nt_tiles;
  // Operand A: one buffer with the fragments and scale bytes of every term at these byte
  // offsets; operand B: one buffer with its fragments and scale bytes.
  const uint8_t* a;
  const uint8_t* b;
  uint32_t a_bytes, b_bytes;
  uint32_t a_frag_off[2], a_sc_off[2], b_frag_off, b_sc_off;
  void* Y;        // float32, or bf16 bits when out_bf16
  int64_t ldy;
  int out_bf16;   // store Y as bf16 (round to nearest, ties to even) instead of float32
  int vec_y;      // Y and ldy allow 16-byte stores of four consecutive outputs
  // grid bookkeeping (32-bit: the workgroup count is far below 2^31)
  uint32_t grid_m, grid_n, per_xcd, n_wg;
  // split-K: ksplit workgroups per tile, each over kper K steps, each writing its partial
  // tile (summed by splitk_reduce_kernel)
  uint32_t ksplit;
  int64_t kper;
  float* partial;
};

// Output tile of linear tile index `tile`: tiles run in groups of kGroupRows row tiles;
// within a group, row tiles vary fastest, then column tiles.  A run of consecutive tiles (the
// workgroups resident on one XCD at a time) then covers a compact block of rows and columns
// that share their A row strips and B column strips in that XCD's L2.
constexpr uint32_t kGroupRows = 8;
__device__ __forceinline__ void tile_coords(uint32_t tile, uint32_t grid_m, uint32_t grid_n, uint32_t& wg_m,
                                            uint32_t& wg_n) {
  const uint32_t group = tile / (kGroupRows * grid_n);
  const uint32_t first = group * kGroupRows;
  const uint32_t rows = min(kGroupRows, grid_m - first);
  const uint32_t in = tile - first * grid_n;
  wg_m = first + in % rows;
  wg_n = in / rows;
}

// float32 -> bf16 bits, round to nearest, ties to even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ void store_y(void* Y, int64_t idx, float v, int out_bf16) {
  if (out_bf16) reinterpret_cast<uint16_t*>(Y)[idx] = f32_to_bf16_rne(v);
  else reinterpret_cast<float*>(Y)[idx] = v;
}

// Four consecutive outputs; Y + idx is 16-byte aligned (float32) or 8-byte aligned (bf16).
__device__ __forceinline__ void store_y4(void* Y, int64_t idx, const v4f& v, int out_bf16) {
  if (out_bf16) {
    const uint32_t lo = f32_to_bf16_rne(v[0]) | ((uint32_t)f32_to_bf16_rne(v[1]) << 16);
    const uint32_t hi = f32_to_bf16_rne(v[2]) | ((uint32_t)f32_to_bf16_rne(v[3]) << 16);
    *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(Y) + idx) = make_uint2(lo, hi);
  } else {
    *reinterpret_cast<v4f*>(reinterpret_cast<float*>(Y) + idx) = v;
  }
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  // raw buffer (32-bit dwords, no swizzle); num_records = bytes bounds every access
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

template <int FA, int FB>
__device__ __forceinline__ v16f mfma(const v8i& a, const v8i& b, const v16f& c, int sa, int sb) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, FA, FB, 0, sa, 0, sb);
}

// Buffer load of SZ bytes per lane into LDS: lane l's bytes land at lds + SZ * l.  The lane's
// offset is voff + soff (soff: the wave-uniform K advance); lanes whose voff lies past the
// buffer's num_records read zeros, and a zero-size buffer makes the whole copy read zeros.
template <int SZ>
__device__ __forceinline__ void copy_to_lds(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff, uint32_t soff) {
  if constexpr (SZ == 16) __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)lds, 16, voff, soff, 0, 0);
  else if constexpr (SZ == 12) __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)lds, 12, voff, soff, 0, 0);
  else __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)lds, 4, voff, soff, 0, 0);
}

// s_waitcnt on vmcnt only (expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt field is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier that also waits for this wave's LDS reads (lgkmcnt) but not for its
// outstanding LDS-destination copies (vmcnt is waited for explicitly).  __syncthreads()
// would wait for every outstanding copy; the memory clobber keeps the compiler from moving
// memory accesses across the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int FMT, int WM, int WN, int TM, int TN, int NT, int NS, int KG>
__global__ __launch_bounds__(64 * WM * WN * KG)
__attribute__((amdgpu_waves_per_eu(kSingleSet<FMT, TM, TN> ? 2 : KG)))
void gemm_kernel(GemmParams p) {
  using G = Geo<FMT, WM, WN, TM, TN, NT, NS, KG>;
  static_assert(G::LDS <= 160 * 1024, "a workgroup's LDS is at most 160 KB on gfx950");
  static_assert((NS - 1) * G::JW < 64, "the vmcnt waits must fit the 6-bit counter");
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];

  const uint32_t b = blockIdx.x;
  const uint32_t wgid = (b % kXcds) * p.per_xcd + b / kXcds;
  if (wgid >= p.n_wg) return;
  const uint32_t ntiles = p.grid_m * p.grid_n;
  const uint32_t split = p.ksplit == 1 ? 0u : wgid / ntiles;  // split-major
  const uint32_t tile = wgid - split * ntiles;
  uint32_t wg_m, wg_n;
  tile_coords(tile, p.grid_m, p.grid_n, wg_m, wg_n);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int kg = wave / G::WT, wt = wave % G::WT;             // K group, wave within it
  const int wm = wt % WM, wn = wt / WM;
  const uint32_t T0 = wg_m * G::MTW, N0 = wg_n * G::NTW;
  const uint32_t nkb = (uint32_t)p.nkb;
  const uint32_t kbeg = (uint32_t)(split * p.kper);                    // this split's K steps:
  const uint32_t klen = (uint32_t)min((int64_t)p.kper, p.nkb - kbeg);  // kbeg .. kbeg+klen-1

  // ---- this wave's copy slots: copy jc of a class goes to wave jc % W (gemm_geo.h) ----
  SlotArgs sargs{};
  sargs.a_frag0 = p.a_frag_off[0];
  sargs.a_frag1 = p.a_frag_off[1];
  sargs.a_sc0 = p.a_sc_off[0];
  sargs.a_sc1 = p.a_sc_off[1];
  sargs.b_frag_off = p.b_frag_off;
  sargs.b_sc_off = p.b_sc_off;
  sargs.T0 = T0;
  sargs.N0 = N0;
  sargs.mt = (uint32_t)p.mt_tiles;
  sargs.nt = (uint32_t)p.nt_tiles;
  sargs.nkb = nkb;
  Slot sa[G::XA], sb[G::XB], ss[G::XS];
  bool ss_a[G::XS];  // scale slot reads operand A's buffer
#pragma unroll
  for (int x = 0; x < G::XA; ++x) sa[x] = slot_a<G>(wave, x, lane, sargs);
#pragma unroll
  for (int x = 0; x < G::XB; ++x) sb[x] = slot_b<G>(wave, x, lane, sargs);
#pragma unroll
  for (int x = 0; x < G::XS; ++x) ss[x] = slot_s<G>(wave, x, lane, sargs, ss_a[x]);

  // Copy stage s of this split (its K steps kbeg + s*KG + kk, kk < KG) into stage buffer
  // `buf`; K steps past the split's end copy zeros (through a zero-size buffer).
  const uint32_t nsteps = (klen + KG - 1) / KG;
  auto issue = [&](int buf, uint32_t s) {
    const uint32_t k0 = s * KG;
    const uint32_t kb = kbeg + k0;
    // K steps of this stage inside the split (wave-uniform: it selects scalar descriptors)
    const uint32_t left = __builtin_amdgcn_readfirstlane(k0 < klen ? klen - k0 : 0u);
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.a, p.a_bytes), rb = make_rsrc(p.b, p.b_bytes);
    const __amdgpu_buffer_rsrc_t za = make_rsrc(p.a, 0u), zb = make_rsrc(p.b, 0u);
    auto inside = [&](const Slot& c) { return KG == 1 ? left > 0u : c.kk < left; };
    uint8_t* st = smem + buf * G::STAGE;
#pragma unroll
    for (int x = 0; x < G::XA; ++x)
      copy_to_lds<16>(inside(sa[x]) ? ra : za, st + sa[x].lds, sa[x].voff, kb * G::A_FRAG);
#pragma unroll
    for (int x = 0; x < G::XB; ++x)
      copy_to_lds<G::SZB>(inside(sb[x]) ? rb : zb, st + sb[x].lds, sb[x].voff, kb * G::B_FRAG);
#pragma unroll
    for (int x = 0; x < G::XS; ++x)
      copy_to_lds<4>(inside(ss[x]) ? (ss_a[x] ? ra : rb) : za, st + ss[x].lds, ss[x].voff, kb * 64u);
  };

  v16f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  constexpr bool SB = kSingleSet<FMT, TM, TN>;
  constexpr int TT = TM * TN;
  v16f Pp = {};    // single register set: partial sums of the tile whose fold is pending
  float fp = 0.f;  // and its weight factor 4 + m_w
  // One K step's MFMA operands of this wave, read from an LDS stage.
  struct Frag {
    v8i b[TN];
    int sb[TN];
    v8i a[NT][TM][FMT == 0 ? 1 : 2];  // HiF4: E2M3 hi, lo
    int sa[NT][TM];
  };
  Frag F[2];

  auto read = [&](Frag& f, int buf) {
    const uint8_t* st = smem + buf * G::STAGE + kg * G::BLK;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int lj = wn * TN + j;
      if constexpr (FMT == 0) {
        const v4i x = *reinterpret_cast<const v4i*>(st + G::B_OFF + lj * 1024 + lane * 16);
        f.b[j] = v8i{x[0], x[1], x[2], x[3], 0, 0, 0, 0};
      } else {
        const uint8_t* bb = st + G::B_OFF + lj * G::B_LDS;
        const v4i x = *reinterpret_cast<const v4i*>(bb + lane * 16);  // 12 bytes used
        const v4i y = *reinterpret_cast<const v4i*>(bb + 1024 + lane * 16);
        f.b[j] = v8i{x[0], x[1], x[2], y[0], y[1], y[2], 0, 0};
      }
      f.sb[j] = st[G::SB_OFF + lj * 64 + lane];
    }
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int li = wm * TM + i;
        const uint8_t* a0 = st + (t * G::MTW + li) * G::A_FRAG;
        if constexpr (FMT == 0) {
          const v4i x = *reinterpret_cast<const v4i*>(a0 + lane * 16);
          f.a[t][i][0] = v8i{x[0], x[1], x[2], x[3], 0, 0, 0, 0};
        } else {
          const v4i p0 = *reinterpret_cast<const v4i*>(a0 + lane * 16);
          const v4i p1 = *reinterpret_cast<const v4i*>(a0 + 1024 + lane * 16);
          const v4i p2 = *reinterpret_cast<const v4i*>(a0 + 2048 + lane * 16);
          f.a[t][i][0] = v8i{p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], 0, 0};
          f.a[t][i][1] = v8i{p1[2], p1[3], p2[0], p2[1], p2[2], p2[3], 0, 0};
        }
        f.sa[t][i] = st[G::SA_OFF + (t * G::SAJ * 4 + li) * 64 + lane];
      }
  };

  // Tiles past the edge of the output hold zero operands, so they are computed like the
  // others (their results are never stored) and the MFMAs stay branch-free.  Term-major
  // order keeps the TM x TN independent accumulator chains interleaved.
  auto mma = [&](const Frag& f) {
    if constexpr (FMT == 0) {
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < TM; ++i) {
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

  // HiF4 with one register set (TM x TN > 1): the step's B fragments first, then per row
  // tile its A fragments (both terms, hi and lo) and its TN tiles.  Each tile's partial sums
  // P are folded (acc += (4 + m_w) P) after the next tile's MFMAs are issued, so the fold's
  // VALU work runs under MFMA execution; the last tile's fold is pending across steps.
  auto step_single = [&](int buf) {
    const uint8_t* st = smem + buf * G::STAGE + kg * G::BLK;
    v8i b[TN];
    int sbs[TN];
    float fbs[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int lj = wn * TN + j;
      const uint8_t* bb = st + G::B_OFF + lj * G::B_LDS;
      const v4i x = *reinterpret_cast<const v4i*>(bb + lane * 16);  // 12 bytes used
      const v4i y = *reinterpret_cast<const v4i*>(bb + 1024 + lane * 16);
      b[j] = v8i{x[0], x[1], x[2], y[0], y[1], y[2], 0, 0};
      const int sc = st[G::SB_OFF + lj * 64 + lane];
      sbs[j] = (sc >> 2) + 92;
      fbs[j] = (float)(4 + (sc & 3));
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int li = wm * TM + i;
      v8i a[NT][2];
      int sas[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const uint8_t* a0 = st + (t * G::MTW + li) * G::A_FRAG;
        const v4i p0 = *reinterpret_cast<const v4i*>(a0 + lane * 16);
        const v4i p1 = *reinterpret_cast<const v4i*>(a0 + 1024 + lane * 16);
        const v4i p2 = *reinterpret_cast<const v4i*>(a0 + 2048 + lane * 16);
        a[t][0] = v8i{p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], 0, 0};
        a[t][1] = v8i{p1[2], p1[3], p2[0], p2[1], p2[2], p2[3], 0, 0};
        sas[t] = st[G::SA_OFF + (t * G::SAJ * 4 + li) * 64 + lane] >> 2;
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int x = i * TN + j, xp = x == 0 ? TT - 1 : x - 1, ip = xp / TN, jp = xp % TN;
        v16f Pc;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int h = 0; h < 2; ++h)
            Pc = mfma<2, 3>(a[t][h], b[j], (t == 0 && h == 0) ? v16f{} : Pc, sas[t] + (h == 0 ? 97 : 93), sbs[j]);
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[ip][jp][r] = fmaf(Pp[r], fp, acc[ip][jp][r]);
        Pp = Pc;
        fp = fbs[j];
      }
    }
  };

  if constexpr (SB) {
    // One register set.  Before step k, stages k .. k+NS-2 are in flight.  Step k: wait for
    // this wave's copies of stage k (NS-2 later stages stay outstanding), barrier (stage k is
    // visible to every wave, and every wave has read stage k-1's buffer), refill that buffer
    // with stage k+NS-1, read stage k and run its MFMAs.  Steps past the end multiply zeros.
#pragma unroll
    for (int s = 0; s < NS - 1; ++s) issue(s, (uint32_t)s);
    for (uint32_t k0 = 0; k0 < nsteps; k0 += NS) {
#pragma unroll
      for (int u = 0; u < NS; ++u) {
        const uint32_t k = k0 + u;
        wait_vmcnt<(NS - 2) * G::JW>();
        lds_barrier();
        issue((u + NS - 1) % NS, k + NS - 1);
        step_single(u);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[TM - 1][TN - 1][r] = fmaf(Pp[r], fp, acc[TM - 1][TN - 1][r]);
  } else {
    // Two register sets.  Before step k, stages k+1 .. k+NS-1 are in flight and step k's
    // operands are in registers.  Step k: wait for this wave's copies of stage k+1 (the NS-2
    // later stages stay outstanding), barrier (stage k+1 is visible to every wave, and every
    // wave has read stage k's buffer), refill that buffer with stage k+NS, read stage k+1's
    // operands, run step k's MFMAs.  Steps past the end multiply zeros.  U unrolls the loop
    // so that every buffer and register-set index is a constant.
    constexpr int U = NS % 2 == 0 ? NS : 2 * NS;
#pragma unroll
    for (int s = 0; s < NS; ++s) issue(s, (uint32_t)s);
    wait_vmcnt<(NS - 1) * G::JW>();
    __syncthreads();
    read(F[0], 0);
    for (uint32_t k0 = 0; k0 < nsteps; k0 += U) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t k = k0 + u;
        wait_vmcnt<(NS - 2) * G::JW>();
        lds_barrier();
        issue(u % NS, k + NS);
        read(F[(u + 1) & 1], (u + 1) % NS);
        mma(F[u & 1]);
        __builtin_amdgcn_sched_barrier(0);  // keep step k's MFMAs ahead of step k+1's barrier
      }
    }
  }
  wait_vmcnt<0>();

  if constexpr (KG > 1) {
    // sum the K groups' accumulators in group order: groups 1.. park theirs in LDS, group 0
    // adds them and stores the tile
    __syncthreads();  // every wave is done with the stage buffers
    float* red = reinterpret_cast<float*>(smem);
    constexpr int PER = TM * TN * 16 * 64;  // floats per wave
    if (kg > 0) {
      float* dst = red + ((size_t)(kg - 1) * G::WT + wt) * PER;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) dst[((i * TN + j) * 16 + r) * 64 + lane] = acc[i][j][r];
    }
    __syncthreads();
    if (kg > 0) return;
#pragma unroll
    for (int g = 1; g < KG; ++g) {
      const float* src = red + ((size_t)(g - 1) * G::WT + wt) * PER;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] += src[((i * TN + j) * 16 + r) * 64 + lane];
    }
  }

  if (p.ksplit > 1) {
    // split K: write this split's partial tile in register order (coalesced per wave)
    constexpr int TE = 64 * G::WT * TM * TN * 16;  // floats per tile
    float* part = p.partial + ((size_t)tile * p.ksplit + split) * TE + (size_t)wt * TM * TN * 16 * 64;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) part[((i * TN + j) * 16 + r) * 64 + lane] = acc[i][j][r];
    return;
  }

  // Y through LDS, eight rows at a time: accumulator registers 4q .. 4q+3 of a tile hold its
  // rows 8q .. 8q+7 (lanes 0-31 rows 8q .. 8q+3, lanes 32-63 rows 8q+4 .. 8q+7), so the wave
  // writes those registers of its TN tiles into its own LDS slot as an 8 x (TN x 32) row-major
  // block and reads it back 16 bytes per lane: each store then covers whole row segments of
  // TN x 32 columns, not 32 columns of two rows.  The slot is this wave's alone (K groups: its
  // reduction slot, already consumed; one group: after a barrier that ends every wave's reads
  // of the stage buffers), and one wave's LDS accesses complete in order, so only the
  // compiler needs to be kept from reordering them.
  constexpr int RW = TN * 32;  // floats per staged row
  static_assert(KG > 1 || (size_t)G::W * 8 * RW * 4 <= G::LDS, "staging slots fit the stage buffers");
  if constexpr (KG == 1) __syncthreads();
  float* slot = reinterpret_cast<float*>(smem) + (size_t)wt * (KG > 1 ? TM * TN * 16 * 64 : 8 * RW);
  const int half = lane >> 5, l32 = lane & 31;
  const int64_t col0 = ((int64_t)N0 + wn * TN) * 32;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) slot[(4 * half + e) * RW + j * 32 + l32] = acc[i][j][4 * q + e];
      asm volatile("" ::: "memory");
      const int64_t row0 = ((int64_t)T0 + wm * TM + i) * 32 + 8 * q;
#pragma unroll
      for (int s = 0; s < TN; ++s) {
        const int f = 4 * lane + 256 * s;  // flat float index in the 8 x RW block
        const v4f v = *reinterpret_cast<const v4f*>(slot + f);
        const int64_t row = row0 + f / RW, col = col0 + f % RW;
        if (row < p.M) {
          if (p.vec_y && col + 3 < p.N) {
            store_y4(p.Y, row * p.ldy + col, v, p.out_bf16);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (col + e < p.N) store_y(p.Y, row * p.ldy + col + e, v[e], p.out_bf16);
          }
        }
      }
      asm volatile("" ::: "memory");
    }
}

// Sum the ksplit partial tiles of each output tile in split order (deterministic) and store
// Y.  Partial element e = wave, tile (i, j), accumulator register r, lane -- the gemm_kernel
// register order; workgroup b handles the 1024 elements of one (wave, i, j) of one tile.
template <int WM, int WN, int TM, int TN>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ partial,
                                                            int ksplit, uint32_t grid_m, uint32_t grid_n,
                                                            int64_t M, int64_t N, void* __restrict__ Y,
                                                            int64_t ldy, int out_bf16) {
  constexpr int PARTS = WM * WN * TM * TN, TE = 1024 * PARTS;
  const uint32_t tile = blockIdx.x / PARTS;
  const int part = (int)(blockIdx.x % PARTS);
  uint32_t wg_m, wg_n;
  tile_coords(tile, grid_m, grid_n, wg_m, wg_n);
  const float* src = partial + (size_t)tile * ksplit * TE + part * 1024;
  const int ij = part % (TM * TN), wave = part / (TM * TN);
  const int i = ij / TN, j = ij % TN, wm = wave % WM, wn = wave / WM;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = threadIdx.x + 256 * q;  // register r = e / 64, lane = e % 64
    const int lane = e & 63, r = e >> 6;
    float v = src[e];
    for (int k = 1; k < ksplit; ++k) v += src[(size_t)k * TE + e];
    const int64_t row = ((int64_t)wg_m * WM * TM + wm * TM + i) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    const int64_t col = ((int64_t)wg_n * WN * TN + wn * TN + j) * 32 + (lane & 31);
    if (row < M && col < N) store_y(Y, row * ldy + col, v, out_bf16);
  }
}

template <int FMT, int WM, int WN, int TM, int TN, int NS, int KG = 1>
void launch_cfg(GemmParams p, int n_terms, hipStream_t s) {
  p.grid_m = (uint32_t)((p.mt_tiles + WM * TM - 1) / (WM * TM));
  p.grid_n = (uint32_t)((p.nt_tiles + WN * TN - 1) / (WN * TN));
  p.n_wg = p.grid_m * p.grid_n * p.ksplit;
  p.per_xcd = (p.n_wg + kXcds - 1) / kXcds;
  const dim3 grid(p.per_xcd * kXcds);
  const dim3 block(64 * WM * WN * KG);
  using G2 = Geo<FMT, WM, WN, TM, TN, 2, NS, KG>;
  using G1 = Geo<FMT, WM, WN, TM, TN, 1, NS, KG>;
  if (n_terms > 1)
    launch_timed(gemm_kernel<FMT, WM, WN, TM, TN, 2, NS, KG>, grid, block, (uint32_t)G2::lds_bytes(), s, p);
  else
    launch_timed(gemm_kernel<FMT, WM, WN, TM, TN, 1, NS, KG>, grid, block, (uint32_t)G1::lds_bytes(), s, p);
  if (p.ksplit > 1)
    launch_timed(splitk_reduce_kernel<WM, WN, TM, TN>, dim3(p.grid_m * p.grid_n * WM * WN * TM * TN), dim3(256),
                 0u, s, (const float*)p.partial, (int)p.ksplit, p.grid_m, p.grid_n, p.M, p.N, p.Y, p.ldy,
                 p.out_bf16);
}

// Tile choice (measured on MI355X): a CU holds one or two workgroups (LDS- and
// register-bound), so the workgroup count decides how many rounds the grid takes.
//  - grids too small for 128-row tiles to fill the chip: 64 x 64 tiles in K groups (two or
//    four groups of four waves, see plan()), and for HiF4 with long K (at least 64 steps per
//    split) K split in two when that fills the CUs;
//  - small grids with long K that 64 x 128 tiles already fill: the wide tiles below with the
//    K split in up to eight;
//  - MXFP4 with M >= 512 (7B decode and prefill): 128 x 256 tiles (fewest A re-reads per
//    byte of B), two workgroups per CU;
//  - otherwise: 128 x 192 tiles.  HiF4 always takes these: with one register set they fit
//    two waves per SIMD (two workgroups per CU at NS = 2), which hides the LDS reads and the
//    fold behind the other workgroup's MFMAs; 128 x 256 HiF4 tiles would spill.  When the
//    HiF4 grid has fewer than two workgroups per CU (M = 256 decode), the tile runs as eight
//    waves of 32 x 96 instead, so each SIMD still holds two waves.
enum TileCfg { kSmall = 0, kWide = 1, kMid = 2, kMid8 = 3, kNarrow = 4 };
// output tile rows and columns of each configuration
constexpr int kTileRows[5] = {64, 128, 128, 128, 64}, kTileCols[5] = {64, 256, 192, 192, 128};
constexpr int kCUs = 256;

struct Plan {
  int cfg, ksplit;
  int kg, ns;  // small tiles: K groups and stages
  int64_t kper, tiles;
  size_t partial_bytes;
};

Plan plan(int fmt, int64_t M, int64_t N, int64_t K, bool may_split) {
  const int64_t mt = (M + 31) / 32, nt = (N + 31) / 32, nkb = (K + 63) / 64;
  auto wgs = [&](int64_t bm, int64_t bn) { return ((mt + bm - 1) / bm) * ((nt + bn - 1) / bn); };
  Plan pl{};
  pl.ksplit = 1;
  pl.kper = nkb;
  if (wgs(4, 4) < 240 && may_split && nkb >= 128 && kCUs / wgs(2, 4) >= 2) {
    // small grids with long K (the down projection of a decode batch): 64 x 128 tiles with K
    // split up to four ways; the wider tile reads each activation fragment for twice the
    // columns (measured at m = 256, 11008 -> 2048: MXFP4 24 -> 21 us, HiF4 30 -> 27 us)
    pl.cfg = kNarrow;
    pl.tiles = wgs(2, 4);
    int64_t ks = kCUs / pl.tiles;
    ks = ks > 4 ? 4 : ks;
    pl.ksplit = (int)ks;
    pl.kper = (nkb + ks - 1) / ks;
    pl.partial_bytes = (size_t)pl.tiles * pl.ksplit * (64 * 128) * sizeof(float);
    pl.kg = fmt == 0 ? 1 : 2;
    pl.ns = fmt == 0 ? 4 : 2;
    return pl;
  }
  if (wgs(4, 4) < 240 && may_split && nkb >= 128) {
    // small grids with long K whose 64 x 128 tiles already fill the CUs (the 7B down
    // projection at m = 512): the wide tiles with K split, which read each activation fragment
    // for 2-4x the columns of the 64 x 64 tiles in K groups and each weight fragment for twice
    // the rows (measured at m = 512, 18944 -> 3584: MXFP4 54 -> 45 us as 128 x 256 in four
    // splits; HiF4 146 -> 97 us as 128 x 192 in six splits, two workgroups per CU)
    const bool mx = fmt == 0;
    pl.cfg = mx ? kWide : kMid;
    pl.tiles = mx ? wgs(4, 8) : wgs(4, 6);
    int64_t ks = (mx ? kCUs : 2 * kCUs) / pl.tiles;
    ks = ks < 2 ? 2 : ks > 8 ? 8 : ks;
    pl.ksplit = (int)ks;
    pl.kper = (nkb + ks - 1) / ks;
    pl.partial_bytes = (size_t)pl.tiles * pl.ksplit * (kTileRows[pl.cfg] * kTileCols[pl.cfg]) * sizeof(float);
    pl.kg = 1;
    pl.ns = mx ? 4 : 2;
    return pl;
  }
  if (wgs(4, 4) < 240) {
    // small grids (no K split: the long-K ones that would gain from one take the tiles
    // above, and the backward never splits)
    pl.cfg = kSmall;
    pl.tiles = wgs(2, 2);
    // K groups and stages (measured).  Grids within the CUs: MXFP4 takes four K groups for
    // long K ranges (>= 128 steps per workgroup) and two otherwise, HiF4 two, with four
    // stages.  Grids beyond the CUs, where workgroups share CUs: long K ranges keep their
    // K groups with two stages (MXFP4 at m = 512, K = 18944: 73.0 us with four stages, 68.7
    // with two); shorter ones take one K group (HiF4 at m = 512, 3584 -> 4608: 47 us with
    // two K groups, 35 us with one and two stages; MXFP4: 21.6 us, 19.4 with one and four).
    const bool crowded = pl.tiles * pl.ksplit > kCUs;
    pl.ns = 4;
    if (fmt == 0) {
      pl.kg = pl.kper >= 128 ? 4 : 2;
      if (crowded) {
        if (pl.kg == 4) pl.ns = 2;
        else pl.kg = 1;
      }
    } else {
      pl.kg = 2;
      if (crowded) {
        pl.ns = 2;
        if (pl.kper < 128) pl.kg = 1;
      }
    }
  } else if (fmt == 0 && M < 512) {
    // MXFP4 decode batches with wide N (gate_up at m = 256): 64 x 128 tiles, one K group,
    // four stages (measured: 21.6-22.5 us as 128 x 192 tiles, 20.2-20.4 us)
    pl.cfg = kNarrow;
    pl.tiles = wgs(2, 4);
    pl.kg = 1;
    pl.ns = 4;
  } else {
    const bool wide = M >= 512 && fmt == 0;
    pl.cfg = wide ? kWide : kMid;
    pl.tiles = wide ? wgs(4, 8) : wgs(4, 6);
    pl.kg = 1;
    pl.ns = fmt == 0 ? 4 : 2;  // HiF4's single register set fits two workgroups per CU at two stages
    // HiF4 grids below two workgroups per CU: eight waves per 128 x 192 tile (two per SIMD)
    if (fmt == 1 && pl.tiles < 2 * kCUs) pl.cfg = kMid8;
  }
  return pl;
}

// Launches the configuration of the plan (one of RESQ_GEMM_CONFIGS); false if none matches.
bool launch_plan(const GemmParams& p, int fmt, const Plan& pl, int n_terms, hipStream_t s) {
#define RESQ_GEMM_LAUNCH(F, C, WM, WN, TM, TN, NS, KG)                                  \
  if (fmt == F && pl.cfg == C && pl.ns == NS && pl.kg == KG) {                          \
    launch_cfg<F, WM, WN, TM, TN, NS, KG>(p, n_terms, s);                               \
    return true;                                                                          \
  }
  RESQ_GEMM_CONFIGS(RESQ_GEMM_LAUNCH)
#undef RESQ_GEMM_LAUNCH
  return false;
}

}  // namespace

namespace {
constexpr size_t kOffsetLimit = (size_t)kBad - (1u << 20);  // 32-bit buffer offsets with headroom
size_t al256(size_t x) { return (x + 255) / 256 * 256; }
}  // namespace

bool gemm_supported(int fmt, int64_t M, int64_t N, int64_t K, int n_terms) {
  const int amode = fmt == 0 ? kPackMx : kPackHiA, bmode = fmt == 0 ? kPackMx : kPackHiB;
  const size_t a = (size_t)n_terms * (al256(frag_bytes(amode, M, K)) + al256(frag_scale_bytes(M, K)));
  const size_t b = al256(frag_bytes(bmode, N, K)) + al256(frag_scale_bytes(N, K));
  return a < kOffsetLimit && b < kOffsetLimit;
}

size_t gemm_split_scratch(int fmt, int64_t M, int64_t N, int64_t K) {
  return plan(fmt, M, N, K, true).partial_bytes;
}

void gemm_plan_info(int fmt, int64_t M, int64_t N, int64_t K, bool may_split, int32_t info[4]) {
  const Plan pl = plan(fmt, M, N, K, may_split);
  info[0] = pl.cfg;
  info[1] = pl.ksplit;
  info[2] = pl.kg;
  info[3] = pl.ns;
}

bool launch_gemm(const GemmOperands& op, hipStream_t s) {
  if (op.M == 0 || op.N == 0) return true;
  const int amode = op.fmt == 0 ? kPackMx : kPackHiA, bmode = op.fmt == 0 ? kPackMx : kPackHiB;
  const size_t af = frag_bytes(amode, op.M, op.K), as = frag_scale_bytes(op.M, op.K);
  const size_t bf = frag_bytes(bmode, op.N, op.K), bs = frag_scale_bytes(op.N, op.K);
  if (op.a_bytes >= kOffsetLimit || op.b_bytes >= kOffsetLimit) return false;
  for (int t = 0; t < op.n_terms; ++t)
    if (op.a_frag_off[t] + af > op.a_bytes || op.a_sc_off[t] + as > op.a_bytes) return false;
  if (op.b_frag_off + bf > op.b_bytes || op.b_sc_off + bs > op.b_bytes) return false;
  const Plan pl = plan(op.fmt, op.M, op.N, op.K, op.partial != nullptr);
  GemmParams p{};
  p.ksplit = (uint32_t)pl.ksplit;
  p.kper = pl.kper;
  p.partial = op.partial;
  p.M = op.M; p.N = op.N; p.K = op.K;
  p.nkb = (op.K + 63) / 64;
  p.mt_tiles = (op.M + 31) / 32;
  p.nt_tiles = (op.N + 31) / 32;
  p.a = op.a; p.b = op.b;
  p.a_bytes = (uint32_t)op.a_bytes; p.b_bytes = (uint32_t)op.b_bytes;
  for (int t = 0; t < 2; ++t) {
    const int u = t < op.n_terms ? t : 0;
    p.a_frag_off[t] = (uint32_t)op.a_frag_off[u];
    p.a_sc_off[t] = (uint32_t)op.a_sc_off[u];
  }
  p.b_frag_off = (uint32_t)op.b_frag_off; p.b_sc_off = (uint32_t)op.b_sc_off;
  p.Y = op.Y; p.ldy = op.ldy; p.out_bf16 = op.out_bf16 ? 1 : 0;
  p.vec_y = (reinterpret_cast<uintptr_t>(op.Y) % 16 == 0 && op.ldy % 4 == 0) ? 1 : 0;
  return launch_plan(p, op.fmt, pl, op.n_terms, s);
}

}  // namespace resq
