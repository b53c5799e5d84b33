// Optional per-kernel timing with HIP events recorded on the launch stream.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

namespace resq {

enum ProfKernel {
  kProfResidual = 0, kProfQuantRows, kProfQuantCols, kProfPack, kProfSelect, kProfGemm, kProfDiag,
  kProfMixed, kProfCount
};

// Returns a token for prof_end (negative when profiling is off).  With kernel_events, the
// scope's events are not recorded around the enqueue: launches made through launch_timed
// while the scope is open carry them in their dispatch (start with the first kernel, stop
// with each kernel, so the last one's end stands), and the interval covers the kernels'
// execution only, as a kernel trace measures it.
int prof_begin(int kernel, hipStream_t s, bool kernel_events = false);
void prof_end(int token, hipStream_t s);

// Events of the kernel-events scope open on this thread (null when there is none).
struct KernelEvents {
  hipEvent_t start = nullptr, stop = nullptr;
  bool first = true;
};
KernelEvents* prof_kernel_events();

// hipLaunchKernelGGL, or its event-carrying form inside a kernel-events scope.
template <typename K, typename... Args>
inline void launch_timed(K kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, Args... args) {
  KernelEvents* ev = prof_kernel_events();
  if (ev != nullptr) {
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, ev->first ? ev->start : nullptr, ev->stop, 0u,
                          args...);
    ev->first = false;
  } else {
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
  }
}

// RAII bracket around one or more launches.
struct ProfScope {
  int token;
  hipStream_t s;
  ProfScope(int kernel, hipStream_t st, bool kernel_events = false)
      : token(prof_begin(kernel, st, kernel_events)), s(st) {}
  ~ProfScope() { prof_end(token, s); }
};

}  // namespace resq
