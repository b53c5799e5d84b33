// Per-kernel timing with HIP events (resq_profile_* in resq.h).
#include "profiler.h"

#include <cstring>
#include <mutex>
#include <vector>

#include "resq.h"

namespace resq {
namespace {

struct Rec {
  int kernel;
  hipEvent_t a, b;
};

std::mutex g_mu;
bool g_on = false;
std::vector<Rec> g_recs;             // recorded, not yet folded
std::vector<hipEvent_t> g_free;      // reusable event handles
int64_t g_launches[kProfCount] = {};
double g_ms[kProfCount] = {};

hipEvent_t take_event() {
  if (!g_free.empty()) {
    hipEvent_t e = g_free.back();
    g_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void fold_locked() {
  for (Rec& r : g_recs) {
    float ms = 0.f;
    if (r.a && r.b && hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      g_launches[r.kernel] += 1;
      g_ms[r.kernel] += ms;
    }
    if (r.a) g_free.push_back(r.a);
    if (r.b) g_free.push_back(r.b);
  }
  g_recs.clear();
}

const char* kNames[kProfCount] = {"residual", "quant_rows", "quant_cols", "pack_hif4", "select", "gemm",
                                  "diagnostics", "mixed"};

thread_local KernelEvents t_ev;
thread_local bool t_ev_open = false;

}  // namespace

KernelEvents* prof_kernel_events() { return t_ev_open ? &t_ev : nullptr; }

int prof_begin(int kernel, hipStream_t s, bool kernel_events) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on) return -1;
  if (g_recs.size() > 4096) fold_locked();
  Rec r{kernel, take_event(), take_event()};
  if (kernel_events && r.a && r.b) {
    t_ev = KernelEvents{r.a, r.b, true};
    t_ev_open = true;
  } else if (r.a) {
    hipEventRecord(r.a, s);
  }
  g_recs.push_back(r);
  return (int)g_recs.size() - 1;
}

void prof_end(int token, hipStream_t s) {
  if (token < 0) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (t_ev_open) {
    t_ev_open = false;
    if (!t_ev.first) return;  // the launches carried the events
    // no kernel was launched: an empty interval
    if (token < (int)g_recs.size() && g_recs[token].a) hipEventRecord(g_recs[token].a, s);
  }
  if (token < (int)g_recs.size() && g_recs[token].b) hipEventRecord(g_recs[token].b, s);
}

}  // namespace resq

extern "C" {

int resq_profile_enable(int on) {
  std::lock_guard<std::mutex> lk(resq::g_mu);
  resq::g_on = on != 0;
  return RESQ_OK;
}

void resq_profile_reset(void) {
  std::lock_guard<std::mutex> lk(resq::g_mu);
  resq::fold_locked();
  for (int i = 0; i < resq::kProfCount; ++i) {
    resq::g_launches[i] = 0;
    resq::g_ms[i] = 0.0;
  }
}

int resq_profile_read(const char* name, int64_t* launches, double* total_ms) {
  if (!name) return RESQ_ERR_ARG;
  std::lock_guard<std::mutex> lk(resq::g_mu);
  resq::fold_locked();
  for (int i = 0; i < resq::kProfCount; ++i) {
    if (std::strcmp(name, resq::kNames[i]) == 0) {
      if (launches) *launches = resq::g_launches[i];
      if (total_ms) *total_ms = resq::g_ms[i];
      return RESQ_OK;
    }
  }
  return RESQ_ERR_ARG;
}

}  // extern "C"
