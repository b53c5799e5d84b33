// Histogram helpers shared by the selections (select.hip) and the residual pass (quant.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace resq {

// The element-wise selection's global histogram: 256 exponent bins then 64 mantissa bins per
// copy, kElemHistCopies copies; workgroup b adds into copy b % kElemHistCopies, so the few
// populated bins are not one contended address for every workgroup's atomics.  Readers sum
// the copies.
constexpr int kElemHistBins = 320;
constexpr int kElemHistCopies = 8;

// The element-wise selection's per-workgroup histograms in LDS: kLdsCopies copies of nb bins,
// copy c at c * (nb + 1) (so that the copies of one bin lie in different banks), lane l adding
// into copy l % kLdsCopies with one plain LDS atomic per element.  A counting pass's keys
// fall into a few bins; on one address the atomics of a wave serialize, and the copies cut
// that chain eight-fold (measured: the mantissa pass at m = 512, d = 3584 took 11.2 us with a
// wave-level add that counted the lanes sharing a leader's digit with one atomic, 5.8 us this
// way).  Readers sum the copies.
constexpr int kLdsCopies = 8;
__device__ __forceinline__ void hist_add_copies(uint32_t* h, int nb, uint32_t digit, bool active) {
  if (active) atomicAdd(&h[(threadIdx.x % kLdsCopies) * (nb + 1) + digit], 1u);
}
__device__ __forceinline__ uint32_t hist_sum_copies(const uint32_t* h, int nb, int bin) {
  uint32_t v = 0;
#pragma unroll
  for (int c = 0; c < kLdsCopies; ++c) v += h[c * (nb + 1) + bin];
  return v;
}

}  // namespace resq
