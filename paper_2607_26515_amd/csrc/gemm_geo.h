// Compile-time geometry of the FP4 GEMM (gemm.hip): the LDS image of one K step, the
// assignment of copy instructions to waves, and each copy's source offset and LDS target.
//
// Plain C++17 with constexpr functions only (no HIP types or intrinsics), so that the kernel
// and a host-side check of its stage protocol compile the same code: the check rebuilds every
// wave's copies from these functions, verifies that the copies of one K step fill exactly the
// LDS bytes the waves then read, with the source bytes the reader expects, and replays the
// kernel's issue / wait / barrier / read sequence against the vmcnt and barrier rules.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace resq {

constexpr uint32_t kBad = 0xFFFFFFF0u;  // an offset past every operand: the load returns 0
constexpr int kDumpBytes = 1024;         // LDS target of the padding copies (never read)

// Compile-time geometry of one configuration: FMT 0 MXFP4 / 1 HiF4; WM x WN waves per K group,
// each owning TM x TN 32x32 output tiles; NT activation terms; NS LDS stages; KG K groups.
template <int FMT, int WM, int WN, int TM, int TN, int NT, int NS, int KG>
struct Geo {
  static constexpr int kFmt = FMT, kWM = WM, kWN = WN, kTM = TM, kTN = TN, kNT = NT, kNS = NS, kKG = KG;
  static constexpr int WT = WM * WN;                  // waves per K group
  static constexpr int W = WT * KG;                   // waves
  static constexpr int kThreads = 64 * W;
  static constexpr int MTW = WM * TM, NTW = WN * TN;  // row / column tiles per workgroup
  static constexpr int FA = FMT == 0 ? 16 : 48;       // A lane record bytes (global)
  static constexpr int FB = FMT == 0 ? 16 : 24;       // B lane record bytes (global)
  static constexpr int PA = FA / 16;                  // A: 16-byte planes per fragment
  static constexpr int A_FRAG = 64 * FA, B_FRAG = 64 * FB;  // bytes per fragment (global)
  // LDS bytes per B fragment: a 12-byte copy lands each lane at a 16-byte stride
  static constexpr int B_LDS = FMT == 0 ? 1024 : 2048;
  static constexpr int SAJ = (MTW + 3) / 4;           // scale copies per A term (4 fragments each)
  static constexpr int SBJ = (NTW + 3) / 4;
  // LDS image of one K step: A [term][row tile][plane][64 x 16 B]; B [col tile] one 16-byte
  // plane (MXFP4) or two planes of 12 bytes per lane at a 16-byte stride (HiF4); A scales
  // [term][copy][4 x 64 B]; B scales [copy][4 x 64 B].  A stage holds KG such images (BLK
  // bytes apart), then the padding copies' dump area.
  static constexpr int B_OFF = NT * MTW * A_FRAG;
  static constexpr int SA_OFF = B_OFF + NTW * B_LDS;
  static constexpr int SB_OFF = SA_OFF + NT * SAJ * 256;
  static constexpr int BLK = (SB_OFF + SBJ * 256 + 255) / 256 * 256;
  static constexpr int DUMP_OFF = KG * BLK;  // padding copies
  static constexpr int STAGE = DUMP_OFF + kDumpBytes;
  // copy instructions per K step by class: A fragments (16 B per lane), B fragments (16 B
  // per lane for MXFP4; two 12-byte halves for HiF4), scale bytes of A and B (4 B per lane);
  // per stage KG times that; per wave: the class count rounded up to a multiple of W
  static constexpr int JA1 = NT * MTW * PA, JB1 = FMT == 0 ? NTW : 2 * NTW, JS1 = NT * SAJ + SBJ;
  static constexpr int JA = KG * JA1, JB = KG * JB1, JS = KG * JS1;
  static constexpr int XA = (JA + W - 1) / W, XB = (JB + W - 1) / W, XS = (JS + W - 1) / W;
  static constexpr int JW = XA + XB + XS;
  static constexpr int SZB = FMT == 0 ? 16 : 12;
  // the K groups' accumulators are summed through the (then idle) LDS of the stages
  static constexpr int RED = (KG - 1) * WT * TM * TN * 16 * 64 * 4;
  static constexpr size_t LDS = (size_t)(NS * STAGE > RED ? NS * STAGE : RED);
  static size_t lds_bytes() { return LDS; }
  static_assert(NS >= 2, "at least two stages");
};

// Every configuration the GEMM instantiates, as X(format, tile configuration, WM, WN, TM, TN,
// NS, KG); the tile configurations are 0: 64 x 64, 1: 128 x 256, 2: 128 x 192, 3: 128 x 192
// in eight waves, 4: 64 x 128 (the numbering of resq_gemm_plan).  Each runs with one or two activation
// terms.  launch_gemm dispatches from this list, and the protocol check walks it.
#define RESQ_GEMM_CONFIGS(X)                                                                     \
  X(0, 0, 2, 2, 1, 1, 4, 2) X(0, 0, 2, 2, 1, 1, 4, 4) X(0, 0, 2, 2, 1, 1, 2, 4)                \
  X(0, 0, 2, 2, 1, 1, 4, 1) X(0, 1, 2, 2, 2, 4, 4, 1)                \
  X(1, 0, 2, 2, 1, 1, 4, 2) X(1, 0, 2, 2, 1, 1, 2, 2) X(1, 0, 2, 2, 1, 1, 2, 1)                \
  X(1, 3, 4, 2, 1, 3, 2, 1) X(1, 2, 2, 2, 2, 3, 2, 1) X(0, 4, 2, 2, 1, 2, 4, 1)                \
  X(1, 4, 2, 2, 1, 2, 2, 2)

// HiF4 with more than one tile per wave keeps one register set and runs two waves per SIMD.
template <int FMT, int TM, int TN>
constexpr bool kSingleSet = FMT == 1 && TM * TN > 1;

// One copy instruction of a wave: this lane's source offset at K step 0 (kBad: no source,
// the lane copies zeros) and the stage-relative LDS destination (the dump area for copies
// that only pad the wave's count).  Each K step adds the class's step to the offset through
// the instruction's scalar offset; a K step past the end is copied through a zero-size
// buffer, so it reads zeros.
struct Slot {
  uint32_t voff, lds, kk;  // kk: the copy's K step within the stage
};

// What a wave's copies depend on besides the geometry: the operand arrays' byte offsets in
// their buffers, the workgroup's first row / column tile, the tile counts and K steps.
struct SlotArgs {
  // operand A's arrays of terms 0 and 1 as separate members: an array indexed by the
  // (run-time) term would put the struct in the kernel's private memory
  uint32_t a_frag0, a_frag1, a_sc0, a_sc1, b_frag_off, b_sc_off;
  uint32_t T0, N0, mt, nt, nkb;
  constexpr uint32_t frag_a(int t) const { return t == 0 ? a_frag0 : a_frag1; }
  constexpr uint32_t scale_a(int t) const { return t == 0 ? a_sc0 : a_sc1; }
};

// Copy x of class A (fragments of operand A, 16 bytes per lane) of wave `wave`, lane `lane`:
// copy jc = wave + W x of the stage's JA copies; copy jc covers K step kk, term t, row tile
// i and 16-byte plane q.
template <class G>
constexpr Slot slot_a(int wave, int x, int lane, const SlotArgs& a) {
  const int jc = wave + G::W * x;
  Slot c{kBad, (uint32_t)G::DUMP_OFF, 0u};
  if (jc < G::JA) {
    const int kk = jc / G::JA1, jl = jc % G::JA1;
    const int t = jl / (G::MTW * G::PA), i = (jl / G::PA) % G::MTW, q = jl % G::PA;
    c.voff = a.T0 + i < a.mt ? a.frag_a(t) + ((a.T0 + i) * a.nkb + kk) * G::A_FRAG + lane * G::FA + q * 16
                             : kBad;
    c.lds = (uint32_t)(kk * G::BLK + (t * G::MTW + i) * G::A_FRAG + q * 1024);
    c.kk = (uint32_t)kk;
  }
  return c;
}

// Copy x of class B (fragments of operand B): column tile j, and for HiF4 the 12-byte half q.
template <class G>
constexpr Slot slot_b(int wave, int x, int lane, const SlotArgs& a) {
  const int jc = wave + G::W * x;
  Slot c{kBad, (uint32_t)G::DUMP_OFF, 0u};
  if (jc < G::JB) {
    const int kk = jc / G::JB1, jl = jc % G::JB1;
    const int j = G::kFmt == 0 ? jl : jl / 2, q = G::kFmt == 0 ? 0 : jl % 2;
    c.voff = a.N0 + j < a.nt ? a.b_frag_off + ((a.N0 + j) * a.nkb + kk) * G::B_FRAG + lane * G::FB + q * 12 : kBad;
    c.lds = (uint32_t)(kk * G::BLK + G::B_OFF + j * G::B_LDS + q * 1024);
    c.kk = (uint32_t)kk;
  }
  return c;
}

// Copy x of class S (scale bytes, 4 per lane: 16 lanes per fragment, 4 fragments per copy):
// A scales of term t for row tiles 4 (jl % SAJ) .. +3, then B scales; is_a tells which
// operand's buffer the copy reads.
template <class G>
constexpr Slot slot_s(int wave, int x, int lane, const SlotArgs& a, bool& is_a) {
  const int jc = wave + G::W * x;
  Slot c{kBad, (uint32_t)G::DUMP_OFF, 0u};
  is_a = true;
  if (jc < G::JS) {
    const int kk = jc / G::JS1, jl = jc % G::JS1;
    c.kk = (uint32_t)kk;
    if (jl < G::kNT * G::SAJ) {
      const int t = jl / G::SAJ, i = 4 * (jl % G::SAJ) + lane / 16;
      const bool ok = i < G::MTW && a.T0 + i < a.mt;
      c.voff = ok ? a.scale_a(t) + ((a.T0 + i) * a.nkb + kk) * 64 + (lane % 16) * 4 : kBad;
      c.lds = (uint32_t)(kk * G::BLK + G::SA_OFF + jl * 256);
    } else {
      const int q = jl - G::kNT * G::SAJ, j = 4 * q + lane / 16;
      const bool ok = j < G::NTW && a.N0 + j < a.nt;
      c.voff = ok ? a.b_sc_off + ((a.N0 + j) * a.nkb + kk) * 64 + (lane % 16) * 4 : kBad;
      c.lds = (uint32_t)(kk * G::BLK + G::SB_OFF + q * 256);
      is_a = false;
    }
  }
  return c;
}

}  // namespace resq
