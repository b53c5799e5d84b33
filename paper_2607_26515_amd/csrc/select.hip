// Global selections of the residual sparsity functions (paper Sec. 4.3): S_alpha% over
// channels, S^{32x64}_alpha% over 32-row x 64-column blocks, and an element-wise variant.
//
// Each one ranks items by a key computed from the dense Q(dX) (dequantized values), keeps the
// `keep` largest (floor(count * alpha / 100), the caller's count; alpha = 50 in the paper's
// experiments), and breaks ties by the lowest index:
//   channel j      : sum over rows i = 0, 1, ..., m-1 of value(i, j)^2, float64, in that order
//   block (I, J)   : over the block's rows in order, each row adding its per-scale-block sums
//                    (exact; written by the residual pass) in column order, float64
//   element (i, j) : |value(i, j)| (exact in float32), index i * d + j
// Non-negative IEEE keys order like their bit patterns, so the k-th largest key is found by a
// most-significant-digit-first radix select on the bits (8-bit digits for the float64 channel
// and block keys; exponent then mantissa digits for the element keys), after which the keys
// equal to it are ranked by index.  Pruned codes become the +0 code in place.
#include "kernels.h"
#include "frag.h"
#include "hist.h"

namespace resq {
namespace {

constexpr int kThreads = 256;
constexpr int kSelThreads = 1024;   // single-workgroup select (channel and block keys)
constexpr int kWordsPerThread = 4;  // element-wise passes: 4 code words = 32 elements

// MXFP4: |value| of the 8 elements of one 32-bit code word, as float32 bit patterns (exact,
// denormals included), two per hardware conversion.
__device__ __forceinline__ void mx_word_keys(uint32_t cw, uint32_t scale, uint32_t key[8]) {
  const uint32_t mag = cw & 0x77777777u;  // magnitudes only
  const float sc = mx_scale_f32((int)scale - 127);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float v0, v1;
    mx_value2((mag >> (8 * q)) & 0xFFu, sc, v0, v1);
    key[2 * q] = __float_as_uint(v0);
    key[2 * q + 1] = __float_as_uint(v1);
  }
}

// Scale word of element (row, j): MX E8M0 byte or the HiF4 meta word.
template <int FMT>
__device__ __forceinline__ uint32_t scale_at(const void* scales, int64_t row, int64_t d, int64_t j) {
  if constexpr (FMT == 0) return reinterpret_cast<const uint8_t*>(scales)[row * (d / 32) + j / 32];
  else return reinterpret_cast<const uint32_t*>(scales)[row * (d / 64) + j / 64];
}

// ---------------------------------------------------------------------------------------
// Channel keys.  Workgroup = 16 channels x 64 row chunks: lane l of wave w sums the squares of
// channel l % 16 over row chunk 4w + l / 16 in float64, and the chunk sums are added in chunk
// (row) order.  16 channels per workgroup give d / 16 workgroups, enough to cover the CUs at
// the layer widths of a decode batch.  The result equals the defined row-by-row sum exactly
// whenever no float64 addition of either order rounds: every square v^2 is a multiple of 2^L,
// L = twice the exponent of the lowest set bit of the smallest such v in the channel, so if
// the total is below 2^(L+53) every partial sum, in any order, is a multiple of 2^L below
// 2^(L+53) and thus exact.  The check uses 2^(L+52) to absorb any rounding of the computed
// total; a channel that fails it is summed again row by row in the defined order.
// ---------------------------------------------------------------------------------------
constexpr int kChanThreads = 1024;  // 16 waves
constexpr int kChanPerWg = 16;      // channels per workgroup
constexpr int kNoBit = 1 << 20;      // "no nonzero term yet" for the lowest-bit exponent

template <int FMT>
__device__ __forceinline__ float decode_at(uint32_t cbyte, uint32_t sc, int64_t j) {
  const uint32_t c = (cbyte >> (4 * (j & 1))) & 15u;
  if constexpr (FMT == 0) {
    float v0, v1;
    mx_value2(c, mx_scale_f32((int)sc - 127), v0, v1);
    return v0;
  } else {
    const int p = (int)(j & 63);
    const int b = (int)((sc >> (8 + p / 8)) & 1u) + (int)((sc >> (16 + p / 4)) & 1u);
    return hif4_value(c, (int)(sc & 0xFFu), b);
  }
}

// Exponent of the lowest set bit of a nonzero float32 (subnormals included).
__device__ __forceinline__ int lowest_bit_exp(float v) {
  const uint32_t u = __float_as_uint(v) & 0x7FFFFFFFu;
  const int ef = (int)(u >> 23);
  const uint32_t sig = ef ? ((u & 0x7FFFFFu) | 0x800000u) : u;
  return (ef ? ef - 150 : -149) + __builtin_ctz(sig);
}

template <int FMT>
__global__ __launch_bounds__(kChanThreads) void channel_keys_kernel(const uint8_t* __restrict__ codes,
                                                                    const void* __restrict__ scales,
                                                                    int64_t m, int64_t d,
                                                                    double* __restrict__ keys) {
  constexpr int NW = kChanThreads / 64, NC = NW * (64 / kChanPerWg), U = 8;
  __shared__ double part[NC][kChanPerWg];
  __shared__ int low[NC][kChanPerWg];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane % kChanPerWg, chunk = wave * (64 / kChanPerWg) + lane / kChanPerWg;
  const int64_t j = (int64_t)blockIdx.x * kChanPerWg + c;
  const int64_t per = (m + NC - 1) / NC;
  const int64_t r0 = min((int64_t)chunk * per, m), r1 = min(r0 + per, m);
  auto value = [&](int64_t row) {
    return decode_at<FMT>(codes[row * (d / 2) + j / 2], scale_at<FMT>(scales, row, d, j), j);
  };
  double acc = 0.0;
  int lo = kNoBit;
  if (j < d) {
    for (int64_t r = r0; r < r1; r += U) {
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = r + u < r1 ? value(r + u) : 0.f;  // loads issued together
#pragma unroll
      for (int u = 0; u < U; ++u) {
        acc += (double)v[u] * (double)v[u];  // exact square: at most 6 significant bits in v
        if (v[u] != 0.f) lo = min(lo, 2 * lowest_bit_exp(v[u]));
      }
    }
  }
  part[chunk][c] = acc;
  low[chunk][c] = lo;
  __syncthreads();
  if (threadIdx.x >= kChanPerWg || j >= d) return;  // thread c finishes channel c
  double sum = 0.0;
  lo = kNoBit;
  for (int w = 0; w < NC; ++w) {
    sum += part[w][c];
    lo = min(lo, low[w][c]);
  }
  if (sum != 0.0 && !(sum < ldexp(1.0, lo + 52))) {
    // some addition may round: the defined order, rows 0 .. m-1
    sum = 0.0;
    for (int64_t r = 0; r < m; ++r) {
      const float v = value(r);
      sum += (double)v * (double)v;
    }
  }
  keys[j] = sum;
}

// ---------------------------------------------------------------------------------------
// Block keys: one thread per 32 x 64 block, rows in order, scale blocks in column order.
// ---------------------------------------------------------------------------------------
// Key of block t = (I, J): the per-scale-block sums of squares of its rows, rows in order,
// scale blocks (P per 64 columns) in column order.
template <int P>
__device__ __forceinline__ double block_key(const double* __restrict__ partials, int64_t m, int64_t d, int64_t t) {
  const int64_t nJ = d / 64;
  const int64_t I = (int64_t)((uint64_t)t / (uint64_t)nJ), J = t - I * nJ;
  const int64_t r1 = (32 * I + 32 < m) ? 32 * I + 32 : m;
  const int64_t ld = d / 64 * P;  // scale blocks per row
  double acc = 0.0;
#pragma unroll 1
  for (int h = 0; h < 32; h += 16) {  // 16 rows at a time: their loads issued together
    double v[16][P];
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
      for (int q = 0; q < P; ++q)
        v[i][q] = 32 * I + h + i < r1 ? partials[(32 * I + h + i) * ld + J * P + q] : 0.0;
#pragma unroll
    for (int i = 0; i < 16; ++i)  // rows in order, scale blocks in column order
#pragma unroll
      for (int q = 0; q < P; ++q)
        if (32 * I + h + i < r1) acc += v[i][q];
  }
  return acc;
}

template <int FMT>
__global__ __launch_bounds__(kThreads) void block_keys_kernel(const double* __restrict__ partials,
                                                              int64_t m, int64_t d,
                                                              double* __restrict__ keys) {
  const int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (t < ((m + 31) / 32) * (d / 64)) keys[t] = block_key<FMT == 0 ? 2 : 1>(partials, m, d, t);
}

// ---------------------------------------------------------------------------------------
// Workgroup-wide exclusive scan of one uint32 per thread (any multiple of 64 threads).
// ---------------------------------------------------------------------------------------
template <int NT, typename T = uint32_t>
__device__ __forceinline__ T block_exclusive_scan(T v, T* wsum, T& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  T x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const T y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  T before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    const T s = wsum[w];
    if (w < wave) before += s;
    all += s;
  }
  __syncthreads();
  total = all;
  return before + x - v;
}

// Radix digit choice over an LDS histogram of nb <= NT bins: the digit holding the k-th
// largest key (k >= 1; k = 0 picks the top digit) and k's rank among the keys with that digit.
// A suffix scan over the bins runs on all threads; every thread of the block must call this,
// and all read the result from out[0] (digit) and out[1] (rank) after it returns.
template <int NT>
__device__ __forceinline__ void choose_digit(const uint32_t* hist, int nb, uint32_t k,
                                             uint32_t* wsum, uint32_t* out) {
  const int tid = threadIdx.x;
  const uint32_t v = tid < nb ? hist[nb - 1 - tid] : 0u;  // bins from the top down
  uint32_t total;
  const uint32_t above = block_exclusive_scan<NT>(v, wsum, total);  // keys in higher bins
  if (tid < nb && ((above < k && k <= above + v) || (k == 0 && tid == 0))) {
    out[0] = (uint32_t)(nb - 1 - tid);
    out[1] = k - above;
  }
  __syncthreads();
}

// Radix digit choice by one wave over a 256-bin histogram (hist.h copies, summed here): the
// digit holding the k-th largest key (k >= 1; k = 0 picks the top digit), k's rank among the
// keys with that digit, and that digit's count, to out[0..2].  Lane l holds bins 255 - 4l ..
// 252 - 4l.
__device__ __forceinline__ void choose_digit_wave(const uint32_t* hist, uint32_t k, uint32_t* out) {
  const int lane = threadIdx.x & 63;
  uint32_t v[4], sum = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[e] = hist_sum_copies(hist, 256, 255 - 4 * lane - e);
    sum += v[e];
  }
  uint32_t incl = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  uint32_t above = incl - sum;  // keys in higher bins
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if ((above < k && k <= above + v[e]) || (k == 0 && lane == 0 && e == 0)) {
      out[0] = (uint32_t)(255 - 4 * lane - e);
      out[1] = k - above;
      out[2] = v[e];
    }
    above += v[e];
  }
}


// ---------------------------------------------------------------------------------------
// Single-workgroup top-k over n float64 keys -> bit mask (bit b of byte i = item 8i + b).
// Thread t holds keys t, t + 1024, ... in registers (KPT of them: n <= 1024 KPT), loaded once
// with coalesced loads.  The threshold's ties are ranked in index order from a table of
// per-slot, per-wave tie counts that one wave scans.
// ---------------------------------------------------------------------------------------
// launch_top takes the smallest instantiation that holds the keys, so that a pass over a few
// thousand keys is not a walk over many mostly empty slots.
constexpr int kKeysPerThread = 20;  // the largest: n <= 20480 (channels of d <= 20480)

// BP = 0: the keys are read from `keys`; BP = 1 / 2 (one key per thread): they are the block
// keys, summed from `partials` (BP scale blocks per 64 columns) at load.
template <int KPT, int BP>
__global__ __launch_bounds__(kSelThreads) void select_top_kernel(const uint64_t* __restrict__ keys,
                                                                 const double* __restrict__ partials,
                                                                 int64_t m, int64_t d, int64_t n, int64_t k,
                                                                 uint8_t* __restrict__ bits,
                                                                 uint8_t* __restrict__ bits_copy) {
  static_assert(BP == 0 || KPT == 1, "block keys are summed at load one per thread");
  constexpr int kKeysPerThread = KPT;
  constexpr int NW = kSelThreads / 64;
  constexpr int HW = kLdsCopies * 257;  // one pass's histogram: hist.h copies of 256 bins
  __shared__ uint32_t hists[2][HW];  // pass p counts into hists[p & 1] while the other is cleared
  __shared__ uint32_t ch[3];
  __shared__ uint32_t tcnt[kKeysPerThread][NW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint64_t kr[kKeysPerThread];
#pragma unroll
  for (int q = 0; q < kKeysPerThread; ++q) {
    const int64_t i = (int64_t)q * kSelThreads + tid;
    if constexpr (BP == 0) kr[q] = i < n ? keys[i] : 0;
    else kr[q] = i < n ? (uint64_t)__double_as_longlong(block_key<BP>(partials, m, d, i)) : 0;
  }
  __shared__ uint64_t found;
  // Candidates: once the keys that share the threshold's digits so far fit one per thread,
  // they are gathered into LDS (in any order: the passes only count them) and the remaining
  // passes read one slot instead of KPT.
  __shared__ uint64_t cand[kSelThreads];
  __shared__ uint32_t ncand;
  const uint64_t below = (1ull << lane) - 1ull;  // lanes before this one
  bool compact = false;
  uint32_t nc = 0;
  // Bits on which all keys agree decide nothing: the OR and AND of the keys bound the digit
  // passes to the byte-aligned span [s_bot, s_top + 8) holding every differing bit (the first
  // pass then splits the keys instead of finding them all in one bin); above it lies the
  // prefix of every key, below it the tail of every key.
  __shared__ uint64_t red_or[NW], red_and[NW];
  uint64_t kor = 0, kand = ~0ull;
#pragma unroll
  for (int q = 0; q < kKeysPerThread; ++q) {
    const int64_t i = (int64_t)q * kSelThreads + tid;
    if (i < n) { kor |= kr[q]; kand &= kr[q]; }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    kor |= __shfl_xor(kor, off, 64);
    kand &= __shfl_xor(kand, off, 64);
  }
  if (lane == 0) { red_or[wave] = kor; red_and[wave] = kand; }
  __syncthreads();
  kor = 0; kand = ~0ull;
#pragma unroll
  for (int w = 0; w < NW; ++w) { kor |= red_or[w]; kand &= red_and[w]; }
  const uint64_t diff = kor ^ kand;  // bits that differ between some two keys
  const int s_top = diff ? (63 - __builtin_clzll(diff)) / 8 * 8 : 0;
  const int s_bot = diff ? __builtin_ctzll(diff) / 8 * 8 : 8;  // no pass when all keys are equal
  const uint64_t above = s_top + 8 < 64 ? ~((1ull << (s_top + 8)) - 1ull) : 0ull;
  uint64_t prefix = kand & above, mask = above;
  uint32_t krem = (uint32_t)k;
  bool single = false;
  for (int i = tid; i < 2 * HW; i += kSelThreads) hists[i / HW][i % HW] = 0;
  __syncthreads();
  // Two barriers per pass: after the counts, and after the digit choice (which one wave makes
  // with a wave scan, while other threads clear the next pass's histogram).
  int pass = 0;
  for (int shift = s_top; shift >= s_bot; shift -= 8, ++pass) {
    uint32_t* hist = hists[pass & 1];
    if (compact) {
      const uint64_t c = tid < (int)nc ? cand[tid] : 0;
      hist_add_copies(hist, 256, (uint32_t)((c >> shift) & 255u), tid < (int)nc && (c & mask) == prefix);
    } else {
#pragma unroll
      for (int q = 0; q < kKeysPerThread; ++q) {
        const int64_t i = (int64_t)q * kSelThreads + tid;
        hist_add_copies(hist, 256, (uint32_t)((kr[q] >> shift) & 255u), i < n && (kr[q] & mask) == prefix);
      }
    }
    __syncthreads();
    if (wave == 0) {
      choose_digit_wave(hist, krem, ch);
    } else {
      for (int i = tid - 64; i < HW; i += kSelThreads - 64)
        hists[(pass + 1) & 1][i] = 0;  // read by no one since the previous pass's choice
    }
    __syncthreads();
    prefix |= (uint64_t)ch[0] << shift;
    krem = ch[1];
    mask |= (uint64_t)255 << shift;
    const uint32_t in_bin = ch[2];  // keys sharing the threshold's digits so far
    if (in_bin == 1 && shift > s_bot) {
      // a single key has this prefix: it is the threshold (krem = 1), no further digit needed
      if (compact) {
        if (tid < (int)nc && (cand[tid] & mask) == prefix) found = cand[tid];
      } else {
#pragma unroll
        for (int q = 0; q < kKeysPerThread; ++q) {
          const int64_t i = (int64_t)q * kSelThreads + tid;
          if (i < n && (kr[q] & mask) == prefix) found = kr[q];
        }
      }
      __syncthreads();
      prefix = found;
      single = true;
      break;
    }
    if (KPT > 1 && !compact && in_bin <= (uint32_t)kSelThreads && shift > s_bot) {
      if (tid == 0) ncand = 0;
      __syncthreads();
#pragma unroll
      for (int q = 0; q < kKeysPerThread; ++q) {
        const int64_t i = (int64_t)q * kSelThreads + tid;
        const bool c = i < n && (kr[q] & mask) == prefix;
        const uint64_t b = __ballot(c);
        uint32_t base = 0;
        if (lane == 0 && b) base = atomicAdd(&ncand, (uint32_t)__popcll(b));
        base = __shfl(base, 0, 64);
        if (c) cand[base + (uint32_t)__popcll(b & below)] = kr[q];
      }
      __syncthreads();
      nc = ncand;
      compact = true;
    }
  }
  // threshold key (the common tail completes it); krem of its ties are kept, in index order
  const uint64_t T = single ? prefix : (prefix | (kand & ((1ull << s_bot) - 1ull)));
  uint64_t tb[kKeysPerThread];  // tie ballots per slot
#pragma unroll
  for (int q = 0; q < kKeysPerThread; ++q) {
    const int64_t i = (int64_t)q * kSelThreads + tid;
    tb[q] = __ballot(i < n && kr[q] == T);
    if (lane == 0) tcnt[q][wave] = (uint32_t)__popcll(tb[q]);
  }
  __syncthreads();
  // exclusive prefix of the tie counts in index order (slot-major, then wave), by wave 0
  constexpr int NTC = kKeysPerThread * NW, PL = (NTC + 63) / 64;
  if (wave == 0) {
    uint32_t* flat = &tcnt[0][0];
    uint32_t v[PL], sum = 0;
#pragma unroll
    for (int e = 0; e < PL; ++e) {
      v[e] = lane * PL + e < NTC ? flat[lane * PL + e] : 0u;
      sum += v[e];
    }
    uint32_t incl = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(incl, o, 64);
      if (lane >= o) incl += y;
    }
    uint32_t run = incl - sum;
#pragma unroll
    for (int e = 0; e < PL; ++e) {
      if (lane * PL + e < NTC) flat[lane * PL + e] = run;
      run += v[e];
    }
  }
  __syncthreads();
  // keep bits: a wave's 64 keys are 8 whole bytes; wave-uniform stores of 8 bytes where the
  // keys and the pointer allow it, else one byte per 8 lanes
  const bool wide = ((uintptr_t)bits % 8 == 0) && (bits_copy == nullptr || (uintptr_t)bits_copy % 8 == 0);
#pragma unroll
  for (int q = 0; q < kKeysPerThread; ++q) {
    const int64_t i0 = (int64_t)q * kSelThreads + wave * 64, i = i0 + lane;
    if (i0 >= n) continue;  // wave-uniform
    const bool in = i < n, tie = ((tb[q] >> lane) & 1ull) != 0;
    const uint32_t rank = tie ? tcnt[q][wave] + (uint32_t)__popcll(tb[q] & below) : 0u;
    const bool keep = in && (kr[q] > T || (tie && rank < krem));
    const uint64_t bal = __ballot(keep);
    if (wide && i0 + 64 <= n) {
      if (lane == 0) {
        *reinterpret_cast<uint64_t*>(bits + (i0 >> 3)) = bal;
        if (bits_copy) *reinterpret_cast<uint64_t*>(bits_copy + (i0 >> 3)) = bal;
      }
    } else if ((lane & 7) == 0 && in) {
      const uint8_t byte = (uint8_t)(bal >> lane);
      bits[i >> 3] = byte;
      if (bits_copy) bits_copy[i >> 3] = byte;
    }
  }
}

// ---------------------------------------------------------------------------------------
// The same top-k for more keys than the registers hold (n > kKeysPerThread * kSelThreads):
// each radix pass streams the keys from global memory (they stay in L2), and the threshold's
// ties are ranked in index order chunk by chunk (1024 consecutive keys per chunk, one per
// thread, a workgroup scan per chunk).  One workgroup, so no cross-workgroup protocol.
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(kSelThreads) void select_top_stream_kernel(const uint64_t* __restrict__ keys,
                                                                        int64_t n, int64_t k,
                                                                        uint8_t* __restrict__ bits,
                                                                        uint8_t* __restrict__ bits_copy) {
  constexpr int NW = kSelThreads / 64;
  __shared__ uint32_t hc[kLdsCopies * 257];  // hist.h copies of the pass's 256 bins
  __shared__ uint32_t hist[256];             // their sums
  __shared__ uint32_t ch[2];
  __shared__ uint32_t wsum[NW];
  __shared__ uint64_t found;
  const int tid = threadIdx.x, lane = tid & 63;
  uint64_t prefix = 0, mask = 0;
  uint32_t krem = (uint32_t)k;
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int i = tid; i < kLdsCopies * 257; i += kSelThreads) hc[i] = 0;
    __syncthreads();
    for (int64_t base = 0; base < n; base += kSelThreads) {
      const int64_t i = base + tid;
      const uint64_t key = i < n ? keys[i] : 0;
      hist_add_copies(hc, 256, (uint32_t)((key >> shift) & 255u), i < n && (key & mask) == prefix);
    }
    __syncthreads();
    if (tid < 256) hist[tid] = hist_sum_copies(hc, 256, tid);
    __syncthreads();
    choose_digit<kSelThreads>(hist, 256, krem, wsum, ch);
    prefix |= (uint64_t)ch[0] << shift;
    krem = ch[1];
    mask |= (uint64_t)255 << shift;
    const uint32_t in_bin = hist[ch[0]];
    __syncthreads();
    if (in_bin == 1 && shift > 0) {
      // a single key has this prefix: it is the threshold
      for (int64_t base = 0; base < n; base += kSelThreads) {
        const int64_t i = base + tid;
        if (i < n && (keys[i] & mask) == prefix) found = keys[i];
      }
      __syncthreads();
      prefix = found;
      break;
    }
  }
  const uint64_t T = prefix;
  uint32_t seen = 0;  // ties in earlier chunks
  for (int64_t base = 0; base < n; base += kSelThreads) {
    const int64_t i = base + tid;
    const bool in = i < n;
    const uint64_t key = in ? keys[i] : 0;
    const bool tie = in && key == T;
    uint32_t total;
    const uint32_t rank = seen + block_exclusive_scan<kSelThreads>(tie ? 1u : 0u, wsum, total);
    const bool keep = in && (key > T || (tie && rank < krem));
    const uint64_t bal = __ballot(keep);
    if ((lane & 7) == 0 && in) {
      const uint8_t byte = (uint8_t)(bal >> lane);
      bits[i >> 3] = byte;
      if (bits_copy) bits_copy[i >> 3] = byte;
    }
    seen += total;
  }
}

void launch_top(const double* keys, int64_t n, int64_t k, uint8_t* bits, uint8_t* bits_copy, hipStream_t s) {
  const uint64_t* kk = (const uint64_t*)keys;
#define RESQ_TOP(KPT)                                                                                \
  if (n <= (int64_t)(KPT) * kSelThreads) {                                                          \
    hipLaunchKernelGGL((select_top_kernel<KPT, 0>), dim3(1), dim3(kSelThreads), 0, s, kk, (const double*)nullptr, \
                       (int64_t)0, (int64_t)0, n, k, bits, bits_copy);                                \
    return;                                                                                          \
  }
  RESQ_TOP(1) RESQ_TOP(2) RESQ_TOP(4) RESQ_TOP(8) RESQ_TOP(16) RESQ_TOP(kKeysPerThread)
#undef RESQ_TOP
  hipLaunchKernelGGL(select_top_stream_kernel, dim3(1), dim3(kSelThreads), 0, s, kk, n, k, bits, bits_copy);
}

// Block keys, then the top-k over them.  HiF4 blocks up to one per thread: the top-k sums the
// keys itself (one launch fewer; measured at m = 512, d = 3584: 10.0 us against 4.1 + 6.6 us).
// MXFP4 has two scale blocks per 64 columns, and one workgroup reading twice the partial sums
// takes longer than the separate key launch (12.0 us against 4.2 + 6.2 us).
void launch_block_top(int fmt, const double* partials, int64_t m, int64_t d, int64_t keep, const SelectWs& ws,
                      uint8_t* bits_copy, hipStream_t s) {
  const int64_t nb = ((m + 31) / 32) * (d / 64);
  if (fmt == 1 && nb <= kSelThreads) {
    hipLaunchKernelGGL((select_top_kernel<1, 1>), dim3(1), dim3(kSelThreads), 0, s, (const uint64_t*)nullptr,
                       partials, m, d, nb, keep, ws.group_bits, bits_copy);
    return;
  }
  const dim3 g((unsigned)((nb + kThreads - 1) / kThreads));
  if (fmt == 0) hipLaunchKernelGGL((block_keys_kernel<0>), g, dim3(kThreads), 0, s, partials, m, d, ws.keys);
  else hipLaunchKernelGGL((block_keys_kernel<1>), g, dim3(kThreads), 0, s, partials, m, d, ws.keys);
  launch_top(ws.keys, nb, keep, ws.group_bits, bits_copy, s);
}

// Channel keys of the dense Q(dX), then the top-k over them.
void launch_channel_top(int fmt, const uint8_t* codes, const void* scales, int64_t m, int64_t d, int64_t keep,
                        const SelectWs& ws, uint8_t* bits_copy, hipStream_t s) {
  const dim3 g((unsigned)((d + kChanPerWg - 1) / kChanPerWg));
  if (fmt == 0) hipLaunchKernelGGL((channel_keys_kernel<0>), g, dim3(kChanThreads), 0, s, codes, scales, m, d, ws.keys);
  else hipLaunchKernelGGL((channel_keys_kernel<1>), g, dim3(kChanThreads), 0, s, codes, scales, m, d, ws.keys);
  launch_top(ws.keys, d, keep, ws.group_bits, bits_copy, s);
}

// Apply kept channels (KIND 0) or kept blocks (KIND 1): one thread per code word; grid x
// covers the d/8 words of a row, y the rows (grid-stride).
template <int KIND>
__global__ __launch_bounds__(kThreads) void apply_groups_kernel(uint32_t* __restrict__ codes,
                                                                int64_t m, int64_t d,
                                                                const uint8_t* __restrict__ gbits,
                                                                uint8_t* __restrict__ keep_mask) {
  const int64_t c8 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (c8 >= d / 8) return;
  for (int64_t row = blockIdx.y; row < m; row += gridDim.y) {
    uint32_t kb;
    if constexpr (KIND == 0) {
      kb = gbits[c8];
    } else {
      const int64_t bit = (row / 32) * (d / 64) + c8 / 8;
      kb = ((gbits[bit >> 3] >> (bit & 7)) & 1u) ? 0xFFu : 0u;
    }
    const int64_t w = row * (d / 8) + c8;
    codes[w] &= nibble_mask8(kb);
    if (keep_mask) keep_mask[w] = (uint8_t)kb;
  }
}

// ---------------------------------------------------------------------------------------
// Element-wise 50%: radix select over the float32 |value| patterns of the decoded Q(dX).
// FP4 values of both formats have no set bits below mantissa bit 17 (MXFP4: at most two
// significant bits, subnormal only in bits 21-22; HiF4: k (4+m) < 64 at a normal exponent),
// so two digit passes fix the threshold exactly: the exponent field (bits 23-30, 256 bins),
// then mantissa bits 17-22 (64 bins) among the keys with the chosen exponent.
// hist: [0, 256) exponent counts, [256, 320) mantissa counts.  Each kernel after the first
// recomputes the choice from the histograms, so no workgroup waits for another.
// ---------------------------------------------------------------------------------------
constexpr int kUHist = kElemHistBins;       // hist.h: 256 exponent bins, then 64 mantissa bins
constexpr int kHistCopies = kElemHistCopies;  // hist.h: copies that readers sum

// Threshold ties.  The second pass counts, per workgroup, the keys of the chosen exponent by
// their six mantissa bits; the threshold is one of those 64 patterns and FP4 keys have no
// lower bits, so that table holds every workgroup's tie count for whichever threshold the
// pass's global histogram then fixes.  The counts are also summed per group of kSuper
// workgroups, so that a workgroup finds the ties of all earlier workgroups in
// O(nwg / kSuper + kSuper) reads.  A group's sums are kSuperCopies copies (workgroup w adds
// into copy w % kSuperCopies), so that the atomics of a group's workgroups do not all hit one
// address; with a single group no workgroup reads them, and none are formed.
constexpr int kSuper = 256;
constexpr int kSuperCopies = 8;
constexpr int kMantBins = 64;

__global__ void uzero_kernel(uint32_t* hist, int words) {
  for (int i = threadIdx.x; i < words; i += blockDim.x) hist[i] = 0;
}

// A thread's 32 elements (4 words of codes from word w0, one scale block): the raw codes and
// scale, loaded before the threshold is known so that their latency overlaps its reads, then
// the keys.
struct ThreadWords {
  uint4 cw;
  uint32_t sc;
  int jpos;
};

template <int FMT>
__device__ __forceinline__ ThreadWords thread_words(const uint8_t* codes, const void* scales, int64_t d, int64_t w0) {
  ThreadWords t;
  t.cw = *reinterpret_cast<const uint4*>(codes + 4 * w0);
  const uint32_t e0 = (uint32_t)(8 * w0), row = e0 / (uint32_t)d, j = e0 - row * (uint32_t)d;
  t.sc = scale_at<FMT>(scales, row, d, j);
  t.jpos = FMT == 0 ? 0 : (int)(j & 63);
  return t;
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// HiF4 keys of word Q of a thread's four (its elements 8Q .. 8Q + 7, one level-2 group and two
// level-3 groups): value k (4 + m) 2^(e - 35 - b).  The eight magnitudes k spread to the bytes
// of two dwords, one 16-bit-lane multiply by 4 + m forms four products k (4 + m) <= 49 at once
// (no carry crosses a byte), each byte converts to float32 exactly, and ldexp applies the
// group's 2^(e - 35 - b) (exact: the smallest nonzero value, 4 * 2^-37, is normal).  f2 holds
// 4 + m in both 16-bit lanes, e35 = e - 35; l2 and l3 are the thread's level-2 and level-3
// shift bits, from its first group on.
template <int Q>
__device__ __forceinline__ void hif4_word_keys(uint32_t cw, uint32_t f2, int e35, uint32_t l2, uint32_t l3,
                                               uint32_t key[8]) {
  const uint32_t ta = __builtin_amdgcn_perm(cw, cw, 0x0C010C00u), tb = __builtin_amdgcn_perm(cw, cw, 0x0C030C02u);
  const uint32_t ka = (ta | (ta << 4)) & 0x07070707u, kb = (tb | (tb << 4)) & 0x07070707u;
  const uint32_t pa = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, ka) * __builtin_bit_cast(u16x2, f2));
  const uint32_t pb = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, kb) * __builtin_bit_cast(u16x2, f2));
  const int b2 = (int)((l2 >> Q) & 1u);
  const int ea = e35 - b2 - (int)((l3 >> (2 * Q)) & 1u), eb = e35 - b2 - (int)((l3 >> (2 * Q + 1)) & 1u);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    key[i] = __float_as_uint(ldexpf((float)((pa >> (8 * i)) & 0xFFu), ea));
    key[4 + i] = __float_as_uint(ldexpf((float)((pb >> (8 * i)) & 0xFFu), eb));
  }
}

template <int FMT>
__device__ __forceinline__ void thread_keys(const ThreadWords& t, uint32_t key[32]) {
  if constexpr (FMT == 1) {
    const uint32_t f2 = (4u + (t.sc & 3u)) * 0x00010001u;
    const int e35 = (int)((t.sc >> 2) & 63u) - 35;
    const uint32_t l2 = t.sc >> (8 + t.jpos / 8), l3 = t.sc >> (16 + t.jpos / 4);
    hif4_word_keys<0>(t.cw.x, f2, e35, l2, l3, key);
    hif4_word_keys<1>(t.cw.y, f2, e35, l2, l3, key + 8);
    hif4_word_keys<2>(t.cw.z, f2, e35, l2, l3, key + 16);
    hif4_word_keys<3>(t.cw.w, f2, e35, l2, l3, key + 24);
  } else {
    mx_word_keys(t.cw.x, t.sc, key);
    mx_word_keys(t.cw.y, t.sc, key + 8);
    mx_word_keys(t.cw.z, t.sc, key + 16);
    mx_word_keys(t.cw.w, t.sc, key + 24);
  }
}

// Resolve the threshold from the global histogram (all threads call this; wave 0 reads the
// histogram, summing its copies, and scans it, one barrier for the rest): out[0] = exponent
// digit, out[1] = rank within it; with full, out[2] = threshold key T and out[3] = the number
// of keys equal to T that are kept.  Lane l holds exponent bins 255 - 4l .. 252 - 4l and
// mantissa bin 63 - l, each digit chosen as by a scan from the top bin down.
__device__ __forceinline__ void load_choice(const uint32_t* hist, uint32_t k, bool full, uint32_t* out) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    uint32_t v[4] = {0u, 0u, 0u, 0u}, mv = 0u;
#pragma unroll
    for (int c = 0; c < kHistCopies; ++c) {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += hist[c * kUHist + 255 - 4 * lane - e];
      if (full) mv += hist[c * kUHist + 256 + 63 - lane];
    }
    // exponent digit: the bin holding the k-th largest key (k = 0: the top bin)
    const uint32_t sum = v[0] + v[1] + v[2] + v[3];
    uint32_t incl = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(incl, o, 64);
      if (lane >= o) incl += y;
    }
    uint32_t above = incl - sum, de = 0, ke = 0;
    bool found = false;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if ((above < k && k <= above + v[e]) || (k == 0 && lane == 0 && e == 0)) {
        de = (uint32_t)(255 - 4 * lane - e);
        ke = k - above;
        found = true;
      }
      above += v[e];
    }
    uint64_t who = __ballot(found);
    int src = who ? __ffsll((unsigned long long)who) - 1 : 0;
    de = __shfl(de, src, 64);
    ke = __shfl(ke, src, 64);
    if (full) {
      // mantissa digit among the keys of exponent de, for rank ke
      uint32_t mincl = mv;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(mincl, o, 64);
        if (lane >= o) mincl += y;
      }
      const uint32_t mabove = mincl - mv;
      const bool hit = (mabove < ke && ke <= mabove + mv) || (ke == 0 && lane == 0);
      who = __ballot(hit);
      src = who ? __ffsll((unsigned long long)who) - 1 : 0;
      const uint32_t dm = (uint32_t)(63 - src), krem = __shfl(ke - mabove, src, 64);
      if (lane == 0) {
        out[2] = (de << 23) | (dm << 17);
        out[3] = krem;
      }
    }
    if (lane == 0) {
      out[0] = de;
      out[1] = ke;
    }
  }
  __syncthreads();
}

template <int FMT, int PASS>
__global__ __launch_bounds__(kThreads) void uhist_kernel(const uint8_t* __restrict__ codes,
                                                         const void* __restrict__ scales, int64_t m,
                                                         int64_t d, uint32_t keep,
                                                         uint32_t* __restrict__ hist,
                                                         uint32_t* __restrict__ super_counts,
                                                         uint32_t* __restrict__ tie_counts) {
  constexpr int NB = PASS == 0 ? 256 : 64, OFF = PASS == 0 ? 0 : 256;
  __shared__ uint32_t lc[kLdsCopies * (NB + 1)];  // this workgroup's counts (hist.h copies)
  __shared__ uint32_t ch[4];
  const int tid = threadIdx.x;
  const int64_t w0 = ((int64_t)blockIdx.x * kThreads + tid) * kWordsPerThread;
  const bool in = w0 < m * (d / 8);
  ThreadWords tw{};
  if (in) tw = thread_words<FMT>(codes, scales, d, w0);
  for (int i = tid; i < kLdsCopies * (NB + 1); i += kThreads) lc[i] = 0;
  uint32_t want = 0;
  if constexpr (PASS == 1) {
    load_choice(hist, keep, false, ch);  // its barrier also ends the clearing
    want = ch[0];
  } else {
    __syncthreads();
  }
  uint32_t key[32];
  if (in) thread_keys<FMT>(tw, key);
  else
#pragma unroll
    for (int e = 0; e < 32; ++e) key[e] = 0;
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    if constexpr (PASS == 0) hist_add_copies(lc, NB, key[e] >> 23, in);
    else hist_add_copies(lc, NB, (key[e] >> 17) & 63u, in && (key[e] >> 23) == want);
  }
  __syncthreads();
  for (int b = tid; b < NB; b += kThreads) {
    const uint32_t c = hist_sum_copies(lc, NB, b);  // local bins 0 .. NB-1 (both passes)
    if (c) atomicAdd(&hist[(blockIdx.x % kHistCopies) * kUHist + OFF + b], c);
    if constexpr (PASS == 1) {
      tie_counts[(size_t)blockIdx.x * kMantBins + b] = c;
      if (c && gridDim.x > kSuper)  // integer sums: any order
        atomicAdd(&super_counts[((blockIdx.x / kSuper) * kSuperCopies + blockIdx.x % kSuperCopies) * kMantBins + b], c);
    }
  }
}

// PMODE < 0: prune the codes in place (and write the keep mask).  PMODE >= 0: leave the codes
// and write S(Q(dX)) as fragment-major MFMA records (pack.hip layout, PackMode PMODE) to
// frag / fscale, including the zero records of rows past m (up to a multiple of 32) and of
// the missing half K step when d % 64 == 32.
template <int FMT, int PMODE>
__global__ __launch_bounds__(kThreads) void uapply_kernel(uint8_t* __restrict__ codes,
                                                          const void* __restrict__ scales, int64_t m,
                                                          int64_t d, uint32_t keep,
                                                          const uint32_t* __restrict__ hist,
                                                          const uint32_t* __restrict__ super_counts,
                                                          const uint32_t* __restrict__ tie_counts,
                                                          uint8_t* __restrict__ keep_mask,
                                                          uint8_t* __restrict__ frag,
                                                          uint8_t* __restrict__ fscale) {
  __shared__ uint32_t ch[4];
  __shared__ uint64_t wsum[kThreads / 64];
  const int64_t w0 = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * kWordsPerThread;
  const bool in = w0 < m * (d / 8);
  ThreadWords tw{};
  if (in) tw = thread_words<FMT>(codes, scales, d, w0);
  load_choice(hist, keep, true, ch);
  const uint32_t T = ch[2], krem = ch[3];
  // ties of earlier workgroups: whole groups of kSuper workgroups, then this group's earlier
  // ones, from the second pass's counts of T's mantissa pattern
  const uint32_t tm = (T >> 17) & 63u, sb = blockIdx.x / kSuper;
  uint32_t before = 0;
  for (uint32_t w = threadIdx.x; w < sb * kSuperCopies; w += kThreads) before += super_counts[w * kMantBins + tm];
  for (uint32_t w = sb * kSuper + threadIdx.x; w < blockIdx.x; w += kThreads)
    before += tie_counts[(size_t)w * kMantBins + tm];
  uint32_t key[32];
  uint32_t ties = 0;
  if (in) {
    thread_keys<FMT>(tw, key);
#pragma unroll
    for (int e = 0; e < 32; ++e) ties += key[e] == T;
  }
  // one scan for both: this workgroup's ties in the low half (their exclusive prefix ranks
  // this thread's ties; at most 8192, no carry), the earlier workgroups' in the high half
  // (only their total is needed; at most m d <= 2^31)
  uint64_t total;
  const uint64_t pre = block_exclusive_scan<kThreads, uint64_t>(((uint64_t)before << 32) | ties, wsum, total);
  uint32_t rank = (uint32_t)(total >> 32) + (uint32_t)pre;
  if (!in) return;
  uint32_t kept = 0;  // 32 keep bits
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    bool keep = key[e] > T;
    if (key[e] == T) keep = rank++ < krem;
    kept |= (uint32_t)keep << e;
  }
  uint4* cw = reinterpret_cast<uint4*>(codes + 4 * w0);
  uint4 v = tw.cw;
  v.x &= nibble_mask8(kept & 0xFFu);
  v.y &= nibble_mask8((kept >> 8) & 0xFFu);
  v.z &= nibble_mask8((kept >> 16) & 0xFFu);
  v.w &= nibble_mask8(kept >> 24);
  if constexpr (PMODE < 0) {
    *cw = v;
    if (keep_mask) *reinterpret_cast<uint32_t*>(keep_mask + w0) = kept;
  } else {
    // this thread's 32 elements are one lane record: row `row`, K elements j .. j+31
    const uint32_t e0 = (uint32_t)(8 * w0), row = e0 / (uint32_t)d, j = e0 - row * (uint32_t)d;
    const int64_t nkb = (d + 63) / 64, kb = j / 64;
    const int half = (int)((j / 32) & 1u);
    const uint32_t sc = tw.sc;  // the scale of this thread's block, loaded above
    const int64_t rec = ((int64_t)(row / 32) * nkb + kb) * 64 + (row & 31) + 32 * half;
    store_frag_record<PMODE>(frag, fscale, rec, v, sc, half);
    const uint4 z = make_uint4(0, 0, 0, 0);
    if ((d & 63) == 32 && j + 32 == (uint32_t)d)  // the missing half K step: zero codes, scale 0
      store_frag_record<PMODE>(frag, fscale, rec + 32, z, 0u, 1);
    if (row + 1 == (uint32_t)m)  // rows past m inside the last row tile: zero records
      for (uint32_t r = row + 1; r % 32 != 0; ++r) {
        const int64_t pr = ((int64_t)(r / 32) * nkb + kb) * 64 + (r & 31);
        store_frag_record<PMODE>(frag, fscale, pr + 32 * half, z, 0u, half);
        if ((d & 63) == 32 && j + 32 == (uint32_t)d) store_frag_record<PMODE>(frag, fscale, pr + 32, z, 0u, 1);
      }
  }
}

int64_t unstructured_wgs(int64_t m, int64_t d) {
  const int64_t per = (int64_t)kThreads * kWordsPerThread;
  return (m * (d / 8) + per - 1) / per;
}

// words cleared before an element-wise selection: the histogram copies and the group counts
int64_t hist_words(int64_t m, int64_t d) {
  return (int64_t)kHistCopies * kUHist + (unstructured_wgs(m, d) + kSuper - 1) / kSuper * kSuperCopies * kMantBins;
}

size_t a256(size_t x) { return (x + 255) & ~(size_t)255; }

int64_t n_blocks(int64_t m, int64_t d) { return ((m + 31) / 32) * (d / 64); }

}  // namespace

int64_t select_max_items() { return (int64_t)1 << 31; }

size_t select_ws_bytes(int sparsity, int fmt, int64_t m, int64_t d) {
  (void)fmt;
  switch (sparsity) {
    case 3:  // channel
      return a256((size_t)d * 8) + a256((size_t)(d + 31) / 32 * 4);
    case 4:  // block
      return a256((size_t)n_blocks(m, d) * 8) + a256((size_t)(n_blocks(m, d) + 31) / 32 * 4);
    case 5:  // element-wise
      return a256((size_t)hist_words(m, d) * 4) + a256((size_t)unstructured_wgs(m, d) * kMantBins * 4);
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
    ws.super_counts = ws.hist + kHistCopies * kUHist;
    ws.tie_counts = (uint32_t*)(p + a256((size_t)hist_words(m, d) * 4));
  }
}

void launch_select(int fmt, int sparsity, int64_t m, int64_t d, int64_t keep, uint8_t* qr_codes,
                   const void* qr_scales, const double* partials, uint8_t* keep_mask,
                   uint8_t* group_mask, const SelectWs& ws, hipStream_t s) {
  if (m == 0 || d == 0) return;
  const dim3 gw((unsigned)((d / 8 + kThreads - 1) / kThreads), (unsigned)(m < 65535 ? m : 65535));
  if (sparsity == 3) {
    launch_channel_top(fmt, qr_codes, qr_scales, m, d, keep, ws, group_mask, s);
    hipLaunchKernelGGL((apply_groups_kernel<0>), gw, dim3(kThreads), 0, s,
                       (uint32_t*)qr_codes, m, d, (const uint8_t*)ws.group_bits, keep_mask);
  } else if (sparsity == 4) {
    launch_block_top(fmt, partials, m, d, keep, ws, group_mask, s);
    hipLaunchKernelGGL((apply_groups_kernel<1>), gw, dim3(kThreads), 0, s,
                       (uint32_t*)qr_codes, m, d, (const uint8_t*)ws.group_bits, keep_mask);
  } else if (sparsity == 5) {
    const unsigned nwg = (unsigned)unstructured_wgs(m, d);
    hipLaunchKernelGGL(uzero_kernel, dim3(1), dim3(kThreads), 0, s, ws.hist, (int)hist_words(m, d));
    const uint32_t k = (uint32_t)keep;
#define RESQ_U(F)                                                                                          \
    hipLaunchKernelGGL((uhist_kernel<F, 0>), dim3(nwg), dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, k, ws.hist,  \
                       ws.super_counts, ws.tie_counts);                                                               \
    hipLaunchKernelGGL((uhist_kernel<F, 1>), dim3(nwg), dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, k, ws.hist,  \
                       ws.super_counts, ws.tie_counts);                                                               \
    hipLaunchKernelGGL((uapply_kernel<F, -1>), dim3(nwg), dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, k,         \
                       (const uint32_t*)ws.hist, (const uint32_t*)ws.super_counts, (const uint32_t*)ws.tie_counts,    \
                       keep_mask, nullptr, nullptr);
    if (fmt == 0) { RESQ_U(0) } else { RESQ_U(1) }
#undef RESQ_U
  }
}

void launch_select_frag(int fmt, int sparsity, int64_t m, int64_t d, int64_t keep, uint8_t* qr_codes,
                        const void* qr_scales, const double* partials, const SelectWs& ws,
                        int pack_mode, uint8_t* frag, uint8_t* fscale, hipStream_t s) {
  if (m == 0 || d == 0) return;
  if (sparsity == 3 || sparsity == 4) {
    const bool chan = sparsity == 3;
    const int64_t n = chan ? d : n_blocks(m, d);
    if (chan) {
      launch_channel_top(fmt, qr_codes, qr_scales, m, d, keep, ws, nullptr, s);
    } else {
      if (partials) launch_block_top(fmt, partials, m, d, keep, ws, nullptr, s);
      else launch_top(ws.keys, n, keep, ws.group_bits, nullptr, s);  // keys from the residual pass
    }
    launch_pack(pack_mode, qr_codes, qr_scales, m, d, frag, fscale, s, chan ? 1 : 2, ws.group_bits);
  } else if (sparsity == 5) {
    // the histograms were cleared before the residual pass, which counted the exponent bins
    const unsigned nwg = (unsigned)unstructured_wgs(m, d);
    const uint32_t k = (uint32_t)keep;
#define RESQ_UF(F, P)                                                                                      \
    hipLaunchKernelGGL((uhist_kernel<F, 1>), dim3(nwg), dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, k, ws.hist,  \
                       ws.super_counts, ws.tie_counts);                                                               \
    hipLaunchKernelGGL((uapply_kernel<F, P>), dim3(nwg), dim3(kThreads), 0, s, qr_codes, qr_scales, m, d, k,          \
                       (const uint32_t*)ws.hist, (const uint32_t*)ws.super_counts, (const uint32_t*)ws.tie_counts,    \
                       (uint8_t*)nullptr, frag, fscale);
    if (fmt == 0) { RESQ_UF(0, kPackMx) } else { RESQ_UF(1, kPackHiA) }
#undef RESQ_UF
  }
}

int select_hist_words(int64_t m, int64_t d) { return (int)hist_words(m, d); }

void launch_select_clear(const SelectWs& ws, int64_t m, int64_t d, hipStream_t s) {
  if (m == 0 || d == 0) return;
  hipLaunchKernelGGL(uzero_kernel, dim3(1), dim3(kThreads), 0, s, ws.hist, (int)hist_words(m, d));
}

}  // namespace resq
