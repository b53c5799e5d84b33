// Activation statistics behind the paper's Figs. 2-4 (Sec. 4.2 and Sec. 4.3): zeros of X and
// of Q(X), quantization blocks holding an element above a threshold, and the error S_2:4
// causes on Q(X) and on Q(dX) (sum of the squares it prunes).
//
// One pass reads X once with the lane layout of the residual pass (a lane = 4 consecutive
// elements, the lanes of a block side by side), quantizes X and dX = X - Q(X) (exact in
// float32) and accumulates per lane.  Each workgroup reduces its lanes in a fixed order and
// writes one row of partial statistics to the workspace; one workgroup then adds the rows in
// a fixed order.  Counts are exact; the sums of squares are float64 (every square is exact)
// and the same on every run.
#include "kernels.h"
#include "profiler.h"
#include "quant_core.h"

namespace resq {
namespace {

constexpr int kThreads = 256;
constexpr int kRowGroups = 256;  // grid.y cap: each workgroup then walks m / 256 rows

// Workgroup sum of one double per thread: butterfly within each wave, then the waves in
// order.  Every thread of the block must call this; thread 0 holds the result.
__device__ __forceinline__ double block_sum(double v, double* lds) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  const int wave = threadIdx.x >> 6;
  __syncthreads();  // lds may still be read by a previous call
  if ((threadIdx.x & 63) == 0) lds[wave] = v;
  __syncthreads();
  double t = 0.0;
  if (threadIdx.x == 0)
    for (int w = 0; w < kThreads / 64; ++w) t += lds[w];
  return t;
}

template <int FMT, bool VEC>
__global__ __launch_bounds__(kThreads) void diag_kernel(const uint16_t* __restrict__ X, int64_t m,
                                                        int64_t d, int64_t ldx, float thr,
                                                        double* __restrict__ partials) {
  __shared__ double lds[kThreads / 64];
  constexpr int G = FMT == kMX ? 8 : 16;  // lanes per quantization block
  const int64_t j4 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  uint32_t zx = 0, zq = 0, ob = 0;
  double eq = 0.0, sq = 0.0, er = 0.0, sr = 0.0;
  if (4 * j4 < d) {  // whole blocks drop out together (d is a multiple of the block size)
    for (int64_t row = blockIdx.y; row < m; row += gridDim.y) {
      float v[4];
      const uint16_t* src = X + row * ldx + 4 * j4;
      if constexpr (VEC) {
        const uint2 t = *reinterpret_cast<const uint2*>(src);
        v[0] = bf16_to_f32(t.x & 0xFFFFu); v[1] = bf16_to_f32(t.x >> 16);
        v[2] = bf16_to_f32(t.y & 0xFFFFu); v[3] = bf16_to_f32(t.y >> 16);
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = bf16_to_f32(src[k]);
      }
      const Quad qx = quantize_quad<FMT>(v);
      float r[4], a = 0.f;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        r[k] = v[k] - qx.val[k];  // exact in float32
        a = fmaxf(a, fabsf(v[k]));
        zx += v[k] == 0.f ? 1u : 0u;
        zq += (qx.code[k] & 7u) == 0u ? 1u : 0u;
      }
      const float bmax = group_max<G>(a);
      ob += ((threadIdx.x & (G - 1)) == 0 && bmax > thr) ? 1u : 0u;
      const Quad qr = quantize_quad<FMT>(r);
      const uint32_t kx = keep_2_of_4(qx.code), kr = keep_2_of_4(qr.code);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const double x2 = (double)qx.val[k] * (double)qx.val[k];
        const double r2 = (double)qr.val[k] * (double)qr.val[k];
        eq += x2;
        er += r2;
        sq += ((kx >> k) & 1u) ? 0.0 : x2;
        sr += ((kr >> k) & 1u) ? 0.0 : r2;
      }
    }
  }
  const double vals[7] = {(double)zx, (double)zq, (double)ob, eq, sq, er, sr};
  double* out = partials + ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * 7;
#pragma unroll
  for (int s = 0; s < 7; ++s) {
    const double t = block_sum(vals[s], lds);
    if (threadIdx.x == 0) out[s] = t;
  }
}

// stats = {m d, zeros X, zeros Q(X), blocks, outlier blocks, energy Q(X), S_2:4 error Q(X),
// energy Q(dX), S_2:4 error Q(dX)}; row w of partials is added by thread w % 256 in order.
__global__ __launch_bounds__(kThreads) void diag_finish_kernel(const double* __restrict__ partials,
                                                               int64_t n_rows, double elements,
                                                               double blocks,
                                                               double* __restrict__ stats) {
  __shared__ double lds[kThreads / 64];
  double acc[7] = {0, 0, 0, 0, 0, 0, 0};
  for (int64_t w = threadIdx.x; w < n_rows; w += kThreads)
#pragma unroll
    for (int s = 0; s < 7; ++s) acc[s] += partials[w * 7 + s];
  double tot[7];
#pragma unroll
  for (int s = 0; s < 7; ++s) tot[s] = block_sum(acc[s], lds);
  if (threadIdx.x == 0) {
    stats[0] = elements;
    stats[1] = tot[0];
    stats[2] = tot[1];
    stats[3] = blocks;
    stats[4] = tot[2];
    stats[5] = tot[3];
    stats[6] = tot[4];
    stats[7] = tot[5];
    stats[8] = tot[6];
  }
}

dim3 diag_grid(int64_t m, int64_t d) {
  return dim3((unsigned)((d / 4 + kThreads - 1) / kThreads),
              (unsigned)(m < kRowGroups ? (m > 0 ? m : 1) : kRowGroups));
}

}  // namespace

size_t diag_ws_bytes(int64_t m, int64_t d) {
  if (m <= 0 || d <= 0) return 0;
  const dim3 g = diag_grid(m, d);
  return (size_t)g.x * g.y * 7 * sizeof(double);
}

void launch_diagnostics(int fmt, const uint16_t* X, int64_t m, int64_t d, int64_t ldx, float thr,
                        double* stats, double* partials, hipStream_t s) {
  const int64_t B = fmt == kMX ? 32 : 64;
  int64_t rows = 0;
  if (m > 0 && d > 0) {
    const dim3 g = diag_grid(m, d);
    rows = (int64_t)g.x * g.y;
    const bool vec = ((uintptr_t)X % 8 == 0) && (ldx % 4 == 0);
#define RESQ_DG(F, V) launch_timed(diag_kernel<F, V>, g, dim3(kThreads), 0u, s, X, m, d, ldx, thr, partials)
    if (fmt == kMX) { if (vec) RESQ_DG(kMX, true); else RESQ_DG(kMX, false); }
    else { if (vec) RESQ_DG(kHI, true); else RESQ_DG(kHI, false); }
#undef RESQ_DG
  }
  launch_timed(diag_finish_kernel, dim3(1), dim3(kThreads), 0u, s, (const double*)partials, rows,
               (double)(m * d), (double)(m * (d / B)), stats);
}

}  // namespace resq
