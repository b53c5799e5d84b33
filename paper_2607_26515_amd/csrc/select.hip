// Global selections of the residual sparsity functions (paper Sec. 4.3): S_50% over
// channels, S^{32x64}_50% over 32-row x 64-column blocks, and an element-wise 50% variant.
//
// Each one ranks items by a key computed from the dense Q(dX) (dequantized values), keeps the
// floor(count / 2) largest, and breaks ties by the lowest index:
//   channel j      : sum over rows i = 0, 1, ..., m-1 of value(i, j)^2, float64, in that order
//   block (I, J)   : over the block's rows in order, each row adding its per-scale-block sums
//                    (exact; written by the residual pass) in column order, float64
//   element (i, j) : |value(i, j)| (exact in float32), index i * d + j
// Non-negative IEEE keys order like their bit patterns, so the k-th largest key is found by a
// most-significant-digit-first radix select on the bits (8-bit digits), after which the keys
// equal to it are ranked by index.  Pruned codes become the +0 code in place.
#include "kernels.h"
#include "device_fp4.h"

namespace resq {
namespace {

constexpr int kThreads = 256;
constexpr int kSelThreads = 1024;   // single-workgroup select (channel and block keys)
constexpr int kWordsPerThread = 4;  // element-wise passes: 4 code words = 32 elements

// |value| of the 8 elements of one 32-bit code word, as float32 bit patterns (all values of
// both formats are exact in float32, denormals included).  jpos = position of the word's first
// element inside its scale block.
template <int FMT>
__device__ __forceinline__ void word_keys(uint32_t cw, uint32_t scale, int jpos, uint32_t key[8]) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t c = (cw >> (4 * e)) & 7u;  // magnitude only
    float v;
    if constexpr (FMT == 0) {
      v = mx_value(c, (int)scale - 127);
    } else {
      const int p = jpos + e;
      const int b = (int)((scale >> (8 + p / 8)) & 1u) + (int)((scale >> (16 + p / 4)) & 1u);
      v = hif4_value(c, (int)(scale & 0xFFu), b);
    }
    key[e] = __float_as_uint(v);
  }
}

// Scale word of element (row, j): MX E8M0 byte or the HiF4 meta word.
template <int FMT>
__device__ __forceinline__ uint32_t scale_at(const void* scales, int64_t row, int64_t d, int64_t j) {
  if constexpr (FMT == 0) return reinterpret_cast<const uint8_t*>(scales)[row * (d / 32) + j / 32];
  else return reinterpret_cast<const uint32_t*>(scales)[row * (d / 64) + j / 64];
}

// ---------------------------------------------------------------------------------------
// Channel keys.  Workgroup = 64 channels; its four waves decode 64-row chunks into LDS in
// parallel, then wave 0 adds them row by row (the fixed sequential order).
// ---------------------------------------------------------------------------------------
constexpr int kChunk = 64;

template <int FMT>
__global__ __launch_bounds__(kThreads) void channel_keys_kernel(const uint8_t* __restrict__ codes,
                                                                const void* __restrict__ scales,
                                                                int64_t m, int64_t d,
                                                                double* __restrict__ keys) {
  __shared__ double sq[kChunk][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t j = (int64_t)blockIdx.x * 64 + lane;
  double acc = 0.0;
  for (int64_t r0 = 0; r0 < m; r0 += kChunk) {
    const int rows = (int)((m - r0) < kChunk ? (m - r0) : kChunk);
    for (int rr = wave; rr < rows; rr += kThreads / 64) {
      double v2 = 0.0;
      if (j < d) {
        const int64_t row = r0 + rr;
        const uint32_t c = (codes[row * (d / 2) + j / 2] >> (4 * (j & 1))) & 15u;
        const uint32_t sc = scale_at<FMT>(scales, row, d, j);
        float v;
        if constexpr (FMT == 0) {
          v = mx_value(c, (int)sc - 127);
        } else {
          const int p = (int)(j & 63);
          const int b = (int)((sc >> (8 + p / 8)) & 1u) + (int)((sc >> (16 + p / 4)) & 1u);
          v = hif4_value(c, (int)(sc & 0xFFu), b);
        }
        v2 = (double)v * (double)v;  // exact: at most 6 significant bits in v
      }
      sq[rr][lane] = v2;
    }
    __syncthreads();
    if (wave == 0)
      for (int rr = 0; rr < rows; ++rr) acc += sq[rr][lane];
    __syncthreads();
  }
  if (wave == 0 && j < d) keys[j] = acc;
}

// ---------------------------------------------------------------------------------------
// Block keys: one thread per 32 x 64 block, rows in order, scale blocks in column order.
// ---------------------------------------------------------------------------------------
template <int FMT>
__global__ __launch_bounds__(kThreads) void block_keys_kernel(const double* __restrict__ partials,
                                                              int64_t m, int64_t d,
                                                              double* __restrict__ keys) {
  constexpr int P = FMT == 0 ? 2 : 1;  // scale blocks per 64 columns
  const int64_t nJ = d / 64, nI = (m + 31) / 32;
  const int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (t >= nI * nJ) return;
  const int64_t I = t / nJ, J = t % nJ;
  const int64_t r1 = (32 * I + 32 < m) ? 32 * I + 32 : m;
  const int64_t ld = d / (FMT == 0 ? 32 : 64);
  double acc = 0.0;
  for (int64_t i = 32 * I; i < r1; ++i)
#pragma unroll
    for (int q = 0; q < P; ++q) acc += partials[i * ld + J * P + q];
  keys[t] = acc;
}

// ---------------------------------------------------------------------------------------
// Workgroup-wide exclusive scan of one uint32 per thread (any multiple of 64 threads).
// ---------------------------------------------------------------------------------------
template <int NT>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* wsum, uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    const uint32_t s = wsum[w];
    if (w < wave) before += s;
    all += s;
  }
  __syncthreads();
  total = all;
  return before + x - v;
}

// Radix digit choice over a 256-bin histogram: the digit holding the krem-th largest key
// among those matching the prefix; krem becomes its rank among keys with that digit.
__device__ __forceinline__ void choose_digit(const uint32_t* hist, uint64_t& digit, uint64_t& krem) {
  uint64_t cum = 0;
  int b = 255;
  for (; b > 0; --b) {
    if (cum + hist[b] >= krem) break;
    cum += hist[b];
  }
  digit = (uint64_t)b;
  krem -= cum;
}

// ---------------------------------------------------------------------------------------
// Single-workgroup top-k over n float64 keys -> bit mask (bit b of byte i = item 8i + b).
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(kSelThreads) void select_top_kernel(const uint64_t* __restrict__ keys,
                                                                 int64_t n, int64_t k,
                                                                 uint8_t* __restrict__ bits,
                                                                 uint8_t* __restrict__ bits_copy) {
  __shared__ uint32_t hist[256];
  __shared__ uint64_t s_prefix, s_krem;
  __shared__ uint32_t wsum[kSelThreads / 64];
  const int tid = threadIdx.x;
  uint64_t prefix = 0, mask = 0;
  if (tid == 0) { s_prefix = 0; s_krem = (uint64_t)k; }
  for (int shift = 56; shift >= 0; shift -= 8) {
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    for (int64_t i = tid; i < n; i += kSelThreads) {
      const uint64_t key = keys[i];
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid == 0) {
      uint64_t digit, krem = s_krem;
      choose_digit(hist, digit, krem);
      s_prefix |= digit << shift;
      s_krem = krem;
    }
    __syncthreads();
    prefix = s_prefix;
    mask |= (uint64_t)255 << shift;
  }
  const uint64_t T = prefix, krem = s_krem;  // threshold key; ties of T to keep (in index order)
  // each thread owns a contiguous run of whole mask bytes
  const int64_t nbytes = (n + 7) / 8;
  const int64_t per = (nbytes + kSelThreads - 1) / kSelThreads;
  const int64_t b0 = tid * per, b1 = (b0 + per < nbytes) ? b0 + per : nbytes;
  uint32_t ties = 0;
  for (int64_t i = 8 * b0; i < 8 * b1 && i < n; ++i) ties += keys[i] == T;
  uint32_t total;
  uint64_t rank = block_exclusive_scan<kSelThreads>(ties, wsum, total);
  for (int64_t bi = b0; bi < b1; ++bi) {
    uint32_t byte = 0;
    for (int e = 0; e < 8; ++e) {
      const int64_t i = 8 * bi + e;
      if (i >= n) break;
      const uint64_t key = keys[i];
      bool keep = key > T;
      if (key == T) keep = rank++ < krem;
      byte |= (uint32_t)keep << e;
    }
    bits[bi] = (uint8_t)byte;
    if (bits_copy) bits_copy[bi] = (uint8_t)byte;
  }
}

// Expand 8 keep bits into a nibble mask for one code word.
__device__ __forceinline__ uint32_t nibble_mask(uint32_t kb) {
  uint32_t m = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) m |= ((kb >> e) & 1u) * (0xFu << (4 * e));
  return m;
}

// Apply kept channels (KIND 0) or kept blocks (KIND 1): one thread per code word.
template <int KIND>
__global__ __launch_bounds__(kThreads) void apply_groups_kernel(uint32_t* __restrict__ codes,
                                                                int64_t m, int64_t d,
                                                                const uint8_t* __restrict__ gbits,
                                                                uint8_t* __restrict__ keep_mask) {
  const int64_t w = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (w >= m * (d / 8)) return;
  const int64_t row = w / (d / 8), c8 = w % (d / 8);
  uint32_t kb;
  if constexpr (KIND == 0) {
    kb = gbits[c8];
  } else {
    const int64_t bit = (row / 32) * (d / 64) + (8 * c8) / 64;
    kb = ((gbits[bit >> 3] >> (bit & 7)) & 1u) ? 0xFFu : 0u;
  }
  codes[w] &= nibble_mask(kb);
  if (keep_mask) keep_mask[w] = (uint8_t)kb;
}

// ---------------------------------------------------------------------------------------
// Element-wise 50%: multi-workgroup radix select over float32 |value| bit patterns.
// state (uint32): [0..3] finished-workgroup counters of the four passes, [4] prefix,
// [5] ties of the threshold still to keep; hist: four 256-bin histograms.
// ---------------------------------------------------------------------------------------
__global__ void unstructured_init_kernel(uint32_t* hist, uint32_t* state, uint32_t k) {
  const int t = threadIdx.x;
  for (int i = t; i < 4 * 256; i += blockDim.x) hist[i] = 0;
  if (t < 8) state[t] = t == 5 ? k : 0u;
}

template <int FMT>
__device__ __forceinline__ void thread_keys(const uint8_t* codes, const void* scales, int64_t d,
                                            int64_t w0, uint32_t key[32]) {
  const uint4 cw = *reinterpret_cast<const uint4*>(codes + 4 * w0);
  const int64_t e0 = 8 * w0, row = e0 / d, j = e0 % d;  // 32 elements inside one scale block
  const uint32_t sc = scale_at<FMT>(scales, row, d, j);
  const int jpos = FMT == 0 ? 0 : (int)(j & 63);
  word_keys<FMT>(cw.x, sc, jpos, key);
  word_keys<FMT>(cw.y, sc, jpos + 8, key + 8);
  word_keys<FMT>(cw.z, sc, jpos + 16, key + 16);
  word_keys<FMT>(cw.w, sc, jpos + 24, key + 24);
}

template <int FMT>
__global__ __launch_bounds__(kThreads) void unstructured_hist_kernel(const uint8_t* __restrict__ codes,
                                                                     const void* __restrict__ scales,
                                                                     int64_t m, int64_t d, int pass,
                                                                     uint32_t* __restrict__ hist,
                                                                     uint32_t* __restrict__ state) {
  __shared__ uint32_t lh[256];
  __shared__ bool last;
  const int tid = threadIdx.x;
  lh[tid] = 0;
  __syncthreads();
  const int shift = 24 - 8 * pass;
  const uint32_t mask = pass == 0 ? 0u : (0xFFFFFFFFu << (32 - 8 * pass));
  const uint32_t prefix = state[4];
  const int64_t words = m * (d / 8);
  const int64_t w0 = ((int64_t)blockIdx.x * kThreads + tid) * kWordsPerThread;
  if (w0 < words) {
    uint32_t key[32];
    thread_keys<FMT>(codes, scales, d, w0, key);
#pragma unroll
    for (int e = 0; e < 32; ++e)
      if ((key[e] & mask) == prefix) atomicAdd(&lh[(key[e] >> shift) & 255u], 1u);
  }
  __syncthreads();
  if (lh[tid]) atomicAdd(&hist[pass * 256 + tid], lh[tid]);
  __threadfence();
  __syncthreads();
  if (tid == 0) last = atomicAdd(&state[pass], 1u) == gridDim.x - 1;
  __syncthreads();
  if (!last) return;
  // the last workgroup to finish picks the digit for the next pass
  __threadfence();
  lh[tid] = __hip_atomic_load(&hist[pass * 256 + tid], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (tid == 0) {
    uint64_t digit, krem = state[5];
    choose_digit(lh, digit, krem);
    state[4] = prefix | ((uint32_t)digit << shift);
    state[5] = (uint32_t)krem;
  }
}

// Threshold ties per workgroup (index order = workgroup order, then thread order).
template <int FMT>
__global__ __launch_bounds__(kThreads) void unstructured_ties_kernel(const uint8_t* __restrict__ codes,
                                                                     const void* __restrict__ scales,
                                                                     int64_t m, int64_t d,
                                                                     const uint32_t* __restrict__ state,
                                                                     uint32_t* __restrict__ tie_counts) {
  __shared__ uint32_t wsum[kThreads / 64];
  const uint32_t T = state[4];
  const int64_t words = m * (d / 8);
  const int64_t w0 = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * kWordsPerThread;
  uint32_t ties = 0;
  if (w0 < words) {
    uint32_t key[32];
    thread_keys<FMT>(codes, scales, d, w0, key);
#pragma unroll
    for (int e = 0; e < 32; ++e) ties += key[e] == T;
  }
  uint32_t total;
  block_exclusive_scan<kThreads>(ties, wsum, total);
  if (threadIdx.x == 0) tie_counts[blockIdx.x] = total;
}

// Exclusive scan of the per-workgroup tie counts, in place (one workgroup).
__global__ __launch_bounds__(kSelThreads) void scan_counts_kernel(uint32_t* __restrict__ c, int64_t n) {
  __shared__ uint32_t wsum[kSelThreads / 64];
  __shared__ uint32_t carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int64_t base = 0; base < n; base += kSelThreads) {
    const int64_t i = base + threadIdx.x;
    const uint32_t v = i < n ? c[i] : 0u;
    uint32_t total;
    const uint32_t ex = block_exclusive_scan<kSelThreads>(v, wsum, total);
    const uint32_t cy = carry;
    if (i < n) c[i] = cy + ex;
    __syncthreads();
    if (threadIdx.x == 0) carry = cy + total;
    __syncthreads();
  }
}

template <int FMT>
__global__ __launch_bounds__(kThreads) void unstructured_apply_kernel(uint8_t* __restrict__ codes,
                                                                      const void* __restrict__ scales,
                                                                      int64_t m, int64_t d,
                                                                      const uint32_t* __restrict__ state,
                                                                      const uint32_t* __restrict__ tie_offsets,
                                                                      uint8_t* __restrict__ keep_mask) {
  __shared__ uint32_t wsum[kThreads / 64];
  const uint32_t T = state[4], krem = state[5];
  const int64_t words = m * (d / 8);
  const int64_t w0 = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * kWordsPerThread;
  uint32_t key[32];
  uint32_t ties = 0;
  const bool in = w0 < words;
  if (in) {
    thread_keys<FMT>(codes, scales, d, w0, key);
#pragma unroll
    for (int e = 0; e < 32; ++e) ties += key[e] == T;
  }
  uint32_t total;
  uint32_t rank = tie_offsets[blockIdx.x] + block_exclusive_scan<kThreads>(ties, wsum, total);
  if (!in) return;
  uint32_t kept = 0;  // 32 keep bits
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    bool keep = key[e] > T;
    if (key[e] == T) keep = rank++ < krem;
    kept |= (uint32_t)keep << e;
  }
  uint4* cw = reinterpret_cast<uint4*>(codes + 4 * w0);
  uint4 v = *cw;
  v.x &= nibble_mask(kept & 0xFFu);
  v.y &= nibble_mask((kept >> 8) & 0xFFu);
  v.z &= nibble_mask((kept >> 16) & 0xFFu);
  v.w &= nibble_mask(kept >> 24);
  *cw = v;
  if (keep_mask) *reinterpret_cast<uint32_t*>(keep_mask + w0) = kept;
}

int64_t unstructured_wgs(int64_t m, int64_t d) {
  const int64_t per = (int64_t)kThreads * kWordsPerThread;
  return (m * (d / 8) + per - 1) / per;
}

size_t a256(size_t x) { return (x + 255) & ~(size_t)255; }

int64_t n_blocks(int64_t m, int64_t d) { return ((m + 31) / 32) * (d / 64); }

}  // namespace

size_t select_ws_bytes(int sparsity, int fmt, int64_t m, int64_t d) {
  (void)fmt;
  switch (sparsity) {
    case 3:  // channel
      return a256((size_t)d * 8) + a256((size_t)(d + 31) / 32 * 4);
    case 4:  // block
      return a256((size_t)n_blocks(m, d) * 8) + a256((size_t)(n_blocks(m, d) + 31) / 32 * 4);
    case 5:  // element-wise
      return a256(4 * 256 * 4) + a256(8 * 4) + a256((size_t)unstructured_wgs(m, d) * 4);
    default:
      return 0;
  }
}

void carve_select_ws(void* base, int sparsity, int fmt, int64_t m, int64_t d, SelectWs& ws) {
  (void)fmt;
  ws = SelectWs{};
  char* p = (char*)base;
  if (sparsity == 3 || sparsity == 4) {
    const int64_t n = sparsity == 3 ? d : n_blocks(m, d);
    ws.keys = (double*)p;
    ws.group_bits = (uint8_t*)(p + a256((size_t)n * 8));
  } else if (sparsity == 5) {
    ws.hist = (uint32_t*)p;
    ws.state = (uint32_t*)(p + a256(4 * 256 * 4));
    ws.tie_counts = (uint32_t*)(p + a256(4 * 256 * 4) + a256(8 * 4));
  }
}

void launch_select(int fmt, int sparsity, int64_t m, int64_t d, uint8_t* qr_codes,
                   const void* qr_scales, const double* partials, uint8_t* keep_mask,
                   uint8_t* group_mask, const SelectWs& ws, hipStream_t s) {
  if (m == 0 || d == 0) return;
  const int64_t words = m * (d / 8);
  const unsigned gw = (unsigned)((words + kThreads - 1) / kThreads);
  if (sparsity == 3) {
    const dim3 g((unsigned)((d + 63) / 64));
    if (fmt == 0) hipLaunchKernelGGL((channel_keys_kernel<0>), g, dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, ws.keys);
    else hipLaunchKernelGGL((channel_keys_kernel<1>), g, dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, ws.keys);
    hipLaunchKernelGGL(select_top_kernel, dim3(1), dim3(kSelThreads), 0, s,
                       (const uint64_t*)ws.keys, d, d / 2, ws.group_bits, group_mask);
    hipLaunchKernelGGL((apply_groups_kernel<0>), dim3(gw), dim3(kThreads), 0, s,
                       (uint32_t*)qr_codes, m, d, (const uint8_t*)ws.group_bits, keep_mask);
  } else if (sparsity == 4) {
    const int64_t nb = n_blocks(m, d);
    const dim3 g((unsigned)((nb + kThreads - 1) / kThreads));
    if (fmt == 0) hipLaunchKernelGGL((block_keys_kernel<0>), g, dim3(kThreads), 0, s, partials, m, d, ws.keys);
    else hipLaunchKernelGGL((block_keys_kernel<1>), g, dim3(kThreads), 0, s, partials, m, d, ws.keys);
    hipLaunchKernelGGL(select_top_kernel, dim3(1), dim3(kSelThreads), 0, s,
                       (const uint64_t*)ws.keys, nb, nb / 2, ws.group_bits, group_mask);
    hipLaunchKernelGGL((apply_groups_kernel<1>), dim3(gw), dim3(kThreads), 0, s,
                       (uint32_t*)qr_codes, m, d, (const uint8_t*)ws.group_bits, keep_mask);
  } else if (sparsity == 5) {
    const int64_t nwg = unstructured_wgs(m, d);
    hipLaunchKernelGGL(unstructured_init_kernel, dim3(1), dim3(kThreads), 0, s, ws.hist, ws.state,
                       (uint32_t)(m * d / 2));
    for (int pass = 0; pass < 4; ++pass) {
      if (fmt == 0) hipLaunchKernelGGL((unstructured_hist_kernel<0>), dim3((unsigned)nwg), dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, pass, ws.hist, ws.state);
      else hipLaunchKernelGGL((unstructured_hist_kernel<1>), dim3((unsigned)nwg), dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, pass, ws.hist, ws.state);
    }
    if (fmt == 0) hipLaunchKernelGGL((unstructured_ties_kernel<0>), dim3((unsigned)nwg), dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, (const uint32_t*)ws.state, ws.tie_counts);
    else hipLaunchKernelGGL((unstructured_ties_kernel<1>), dim3((unsigned)nwg), dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, (const uint32_t*)ws.state, ws.tie_counts);
    hipLaunchKernelGGL(scan_counts_kernel, dim3(1), dim3(kSelThreads), 0, s, ws.tie_counts, nwg);
    if (fmt == 0) hipLaunchKernelGGL((unstructured_apply_kernel<0>), dim3((unsigned)nwg), dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, (const uint32_t*)ws.state, (const uint32_t*)ws.tie_counts, keep_mask);
    else hipLaunchKernelGGL((unstructured_apply_kernel<1>), dim3((unsigned)nwg), dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, (const uint32_t*)ws.state, (const uint32_t*)ws.tie_counts, keep_mask);
  }
}

}  // namespace resq
