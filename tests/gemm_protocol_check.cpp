// Host-side check of the FP4 GEMM's LDS stage protocol, for every configuration the kernel
// instantiates (RESQ_GEMM_CONFIGS, one and two activation terms).  It uses the kernel's own
// geometry and copy assignment (gemm_geo.h) and a model of its main loops' event sequence.
//
// 1. Limits: LDS per workgroup within 160 KB; the largest vmcnt wait within the 6-bit field.
// 2. Data flow of one stage: every wave's copies are built from slot_a / slot_b / slot_s; no
//    two copies write the same LDS byte (the padding copies write only the dump area), and
//    every byte a wave reads for its MFMA operands (A planes, B halves, scale bytes) was
//    written by a copy of the same K step from exactly the source byte the reader interprets
//    it as, or comes from a zero source where the tile lies past the edge.
// 3. Schedule: the kernel's sequence of issue / s_waitcnt vmcnt(N) / barrier / LDS read events
//    is replayed for every number of K steps up to a few full unrolls.  Each wave's copies
//    complete in issue order, so vmcnt(N) guarantees all but its newest N copies; a barrier
//    makes what every wave completed before it visible to all, and (with lgkmcnt(0) before
//    it) ends every wave's earlier LDS reads.  A read of buffer b must find the stage it
//    expects as the last one issued into b, completed before the last barrier; an issue into
//    b must come after a barrier that follows every read of b's previous stage.
//
// Usage: gemm_protocol_check [plant]; plant = 1 waits for one copy too few, plant = 2 refills
// a stage before the barrier, plant = 3 moves a padding copy onto an A fragment: each must be
// reported (the test runs them to see that the check can fail).
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "gemm_geo.h"

using namespace resq;

static int g_plant = 0;
static int g_errors = 0;

#define FAIL(...)                   \
  do {                              \
    if (g_errors < 20) {            \
      std::printf("  FAIL: ");      \
      std::printf(__VA_ARGS__);     \
      std::printf("\n");            \
    }                               \
    ++g_errors;                     \
  } while (0)

// Source of an LDS byte: buffer (0 none, 1 A, 2 B, 3 zero) and byte offset.
struct Src {
  int buf = 0;
  int64_t off = 0;
  bool operator==(const Src& o) const { return buf == o.buf && (buf == 3 || off == o.off); }
};

template <class G>
void check_dataflow(const char* name, bool edge) {
  SlotArgs a{};
  a.a_frag0 = 0;
  a.a_frag1 = 1u << 24;
  a.a_sc0 = 1u << 26;
  a.a_sc1 = (1u << 26) + (1u << 22);
  a.b_frag_off = 0;
  a.b_sc_off = 1u << 26;
  a.T0 = 8;
  a.N0 = 16;
  a.nkb = 40;
  // edge: only the workgroup's first row tile and first column tile exist
  a.mt = edge ? a.T0 + 1 : 1u << 20;
  a.nt = edge ? a.N0 + 1 : 1u << 20;
  std::vector<Src> lds(G::STAGE);
  std::vector<int> writes(G::STAGE, 0);
  auto put = [&](const Slot& c, int lane, int bytes, int stride, int buf, const char* cls) {
    if (c.lds == (uint32_t)G::DUMP_OFF && c.voff == kBad) {  // a padding copy
      if (G::DUMP_OFF + stride * 64 > G::STAGE) FAIL("%s %s: padding copy overruns the dump area", name, cls);
      return;
    }
    for (int b = 0; b < bytes; ++b) {
      const int64_t at = (int64_t)c.lds + (int64_t)stride * lane + b;
      if (at < 0 || at >= G::DUMP_OFF) {
        FAIL("%s %s: copy writes LDS byte %lld outside the K-step images", name, cls, (long long)at);
        return;
      }
      ++writes[at];
      lds[at] = c.voff == kBad ? Src{3, 0} : Src{buf, (int64_t)c.voff + b};
    }
  };
  for (int w = 0; w < G::W; ++w)
    for (int lane = 0; lane < 64; ++lane) {
      for (int x = 0; x < G::XA; ++x) {
        Slot c = slot_a<G>(w, x, lane, a);
        if (g_plant == 3 && w == G::W - 1 && x == G::XA - 1 && c.lds == (uint32_t)G::DUMP_OFF) {
          c.lds = 0;  // planted: a padding copy lands on the first A fragment
          c.voff = 0;
        }
        put(c, lane, 16, 16, 1, "A");
      }
      for (int x = 0; x < G::XB; ++x) put(slot_b<G>(w, x, lane, a), lane, G::SZB, 16, 2, "B");
      for (int x = 0; x < G::XS; ++x) {
        bool is_a = true;
        const Slot c = slot_s<G>(w, x, lane, a, is_a);
        put(c, lane, 4, 4, is_a ? 1 : 2, "scale");
      }
    }
  for (int i = 0; i < G::DUMP_OFF; ++i)
    if (writes[i] > 1) {
      FAIL("%s: LDS byte %d written by %d copies", name, i, writes[i]);
      break;
    }
  // the reads of every wave (kernel's read() / step_single(): same addresses)
  auto expect = [&](int64_t at, Src want, const char* what) {
    if (writes[at] != 1) {
      FAIL("%s: %s reads LDS byte %lld that no copy writes", name, what, (long long)at);
      return false;
    }
    if (!(lds[at] == want)) {
      FAIL("%s: %s reads LDS byte %lld holding source (%d, %lld), expected (%d, %lld)", name, what,
           (long long)at, lds[at].buf, (long long)lds[at].off, want.buf, (long long)want.off);
      return false;
    }
    return true;
  };
  for (int wave = 0; wave < G::W; ++wave) {
    const int kg = wave / G::WT, wt = wave % G::WT, wm = wt % G::kWM, wn = wt / G::kWM;
    const int64_t base = (int64_t)kg * G::BLK;
    for (int lane = 0; lane < 64; ++lane) {
      bool ok = true;
      for (int j = 0; j < G::kTN && ok; ++j) {
        const int lj = wn * G::kTN + j;
        const bool in = a.N0 + lj < a.nt;
        const int halves = G::kFmt == 0 ? 1 : 2;
        for (int q = 0; q < halves && ok; ++q)
          for (int b = 0; b < G::SZB && ok; ++b) {
            const int64_t src = (int64_t)a.b_frag_off + ((int64_t)(a.N0 + lj) * a.nkb + kg) * G::B_FRAG +
                                lane * G::FB + q * 12 + b;
            ok = expect(base + G::B_OFF + lj * G::B_LDS + q * 1024 + lane * 16 + b, in ? Src{2, src} : Src{3, 0},
                        "B fragment");
          }
        if (ok) {
          const int64_t src = (int64_t)a.b_sc_off + ((int64_t)(a.N0 + lj) * a.nkb + kg) * 64 + lane;
          ok = expect(base + G::SB_OFF + lj * 64 + lane, in ? Src{2, src} : Src{3, 0}, "B scale");
        }
      }
      for (int t = 0; t < G::kNT && ok; ++t)
        for (int i = 0; i < G::kTM && ok; ++i) {
          const int li = wm * G::kTM + i;
          const bool in = a.T0 + li < a.mt;
          for (int pl = 0; pl < G::PA && ok; ++pl)
            for (int b = 0; b < 16 && ok; ++b) {
              const int64_t src = (int64_t)(t == 0 ? a.a_frag0 : a.a_frag1) + ((int64_t)(a.T0 + li) * a.nkb + kg) * G::A_FRAG +
                                  lane * G::FA + pl * 16 + b;
              ok = expect(base + (t * G::MTW + li) * G::A_FRAG + pl * 1024 + lane * 16 + b,
                          in ? Src{1, src} : Src{3, 0}, "A fragment");
            }
          if (ok) {
            const int64_t src = (int64_t)(t == 0 ? a.a_sc0 : a.a_sc1) + ((int64_t)(a.T0 + li) * a.nkb + kg) * 64 + lane;
            ok = expect(base + G::SA_OFF + (t * G::SAJ * 4 + li) * 64 + lane, in ? Src{1, src} : Src{3, 0},
                        "A scale");
          }
        }
    }
  }
}

// Event model of the main loops (the kernel's loop structure, copied as events).
enum Ev { kIssue, kWait, kBarrier, kRead };
struct Event {
  Ev e;
  int a, b;  // issue: buffer, stage; wait: N; read: buffer, stage
};

template <class G>
std::vector<Event> schedule(int nsteps) {
  constexpr int NS = G::kNS, JW = G::JW;
  std::vector<Event> ev;
  const bool single = kSingleSet<G::kFmt, G::kTM, G::kTN>;
  const int wait_n = (NS - 2) * JW + (g_plant == 1 ? 1 : 0);
  if (single) {
    for (int s = 0; s < NS - 1; ++s) ev.push_back({kIssue, s, s});
    for (int k0 = 0; k0 < nsteps; k0 += NS)
      for (int u = 0; u < NS; ++u) {
        const int k = k0 + u;
        ev.push_back({kWait, wait_n, 0});
        if (g_plant == 2) ev.push_back({kIssue, (u + NS - 1) % NS, k + NS - 1});
        ev.push_back({kBarrier, 0, 0});
        if (g_plant != 2) ev.push_back({kIssue, (u + NS - 1) % NS, k + NS - 1});
        ev.push_back({kRead, u, k});
      }
  } else {
    const int U = NS % 2 == 0 ? NS : 2 * NS;
    for (int s = 0; s < NS; ++s) ev.push_back({kIssue, s, s});
    ev.push_back({kWait, (NS - 1) * JW, 0});
    ev.push_back({kBarrier, 0, 0});
    ev.push_back({kRead, 0, 0});
    for (int k0 = 0; k0 < nsteps; k0 += U)
      for (int u = 0; u < U; ++u) {
        const int k = k0 + u;
        ev.push_back({kWait, wait_n, 0});
        if (g_plant == 2) ev.push_back({kIssue, u % NS, k + NS});
        ev.push_back({kBarrier, 0, 0});
        if (g_plant != 2) ev.push_back({kIssue, u % NS, k + NS});
        ev.push_back({kRead, (u + 1) % NS, k + 1});
      }
  }
  ev.push_back({kWait, 0, 0});   // wait_vmcnt<0>() after the loop
  ev.push_back({kBarrier, 0, 0});  // the K-group reduction's __syncthreads (the end of the kernel otherwise)
  return ev;
}

template <class G>
void check_schedule(const char* name) {
  constexpr int NS = G::kNS, JW = G::JW;
  const int U = kSingleSet<G::kFmt, G::kTM, G::kTN> ? NS : (NS % 2 == 0 ? NS : 2 * NS);
  for (int nsteps = 1; nsteps <= 3 * U + 2; ++nsteps) {
    const auto ev = schedule<G>(nsteps);
    std::vector<int> issued;              // stage of each copy, in issue order (JW per issue)
    int completed = 0;                    // copies known complete (a prefix)
    int visible_below = 0;                // copies complete before the last barrier
    std::vector<int> content(NS, -1);     // stage last issued into each buffer
    std::vector<int> last_read(NS, -1);   // event index of the last read of each buffer
    int last_barrier = -1;
    std::vector<int> stage_end;           // copy count after each stage's issue
    auto stage_done_by = [&](int stage, int copies) {
      return stage < (int)stage_end.size() && stage_end[stage] <= copies;
    };
    for (int i = 0; i < (int)ev.size(); ++i) {
      const Event& e = ev[i];
      if (e.e == kIssue) {
        if (last_read[e.a] > last_barrier)
          FAIL("%s nsteps %d: stage %d is copied into buffer %d before every wave is done reading it", name,
               nsteps, e.b, e.a);
        if (e.b != (int)stage_end.size()) FAIL("%s: stages issued out of order", name);
        for (int c = 0; c < JW; ++c) issued.push_back(e.b);
        stage_end.push_back((int)issued.size());
        content[e.a] = e.b;
      } else if (e.e == kWait) {
        if (e.a < 0 || e.a >= 64) FAIL("%s: vmcnt(%d) outside the 6-bit field", name, e.a);
        const int done = (int)issued.size() - e.a;
        if (done > completed) completed = done;
      } else if (e.e == kBarrier) {
        last_barrier = i;
        visible_below = completed;  // every wave has completed this many of its copies
      } else {
        if (content[e.a] != e.b)
          FAIL("%s nsteps %d: step %d reads buffer %d, which holds stage %d", name, nsteps, e.b, e.a, content[e.a]);
        else if (!stage_done_by(e.b, visible_below))
          FAIL("%s nsteps %d: step %d reads stage %d before every wave's copies of it are complete and a "
               "barrier has followed", name, nsteps, e.b, e.b);
        last_read[e.a] = i;
      }
      if (g_errors > 20) return;
    }
    if (completed != (int)issued.size()) FAIL("%s: copies still outstanding at the end", name);
  }
}

template <class G>
void check_config(const char* name) {
  if (G::LDS > 160 * 1024) FAIL("%s: LDS %zu bytes > 160 KB", name, (size_t)G::LDS);
  if ((G::kNS - 1) * G::JW >= 64) FAIL("%s: vmcnt wait %d beyond the 6-bit field", name, (G::kNS - 1) * G::JW);
  check_dataflow<G>(name, false);
  check_dataflow<G>(name, true);
  check_schedule<G>(name);
}

int main(int argc, char** argv) {
  g_plant = argc > 1 ? std::atoi(argv[1]) : 0;
  int configs = 0;
#define RESQ_CHECK(F, C, WM, WN, TM, TN, NS, KG)                                                          \
  for (int nt = 1; nt <= 2; ++nt) {                                                                       \
    char name[128];                                                                                       \
    std::snprintf(name, sizeof(name), "fmt %d cfg %d %dx%d waves, %dx%d tiles, NS %d, KG %d, %d term(s)", \
                  F, C, WM, WN, TM, TN, NS, KG, nt);                                                      \
    const int before = g_errors;                                                                          \
    if (nt == 1) check_config<Geo<F, WM, WN, TM, TN, 1, NS, KG>>(name);                                   \
    else check_config<Geo<F, WM, WN, TM, TN, 2, NS, KG>>(name);                                           \
    std::printf("%s %s\n", g_errors == before ? "ok  " : "FAIL", name);                                   \
    ++configs;                                                                                            \
  }
  RESQ_GEMM_CONFIGS(RESQ_CHECK)
#undef RESQ_CHECK
  std::printf("%d configurations, %d errors\n", configs, g_errors);
  return g_errors == 0 ? 0 : 1;
}
