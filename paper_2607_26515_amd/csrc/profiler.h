// Optional per-kernel timing with HIP events recorded on the launch stream.
#pragma once

#include <hip/hip_runtime.h>

namespace resq {

enum ProfKernel {
  kProfResidual = 0, kProfQuantRows, kProfQuantCols, kProfPack, kProfSelect, kProfGemm, kProfDiag,
  kProfCount
};

// Returns a token for prof_end (negative when profiling is off).
int prof_begin(int kernel, hipStream_t s);
void prof_end(int token, hipStream_t s);

// RAII bracket around one or more launches.
struct ProfScope {
  int token;
  hipStream_t s;
  ProfScope(int kernel, hipStream_t st) : token(prof_begin(kernel, st)), s(st) {}
  ~ProfScope() { prof_end(token, s); }
};

}  // namespace resq
