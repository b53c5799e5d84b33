// Host-side launchers of the library's HIP kernels (internal; the public ABI is resq.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace resq {

// Residual-path kinds handled inside the quantize pass.
enum ResidMode {
  kResidNone = 0,      // Q(X) only
  kResidIdentity = 1,  // Q(dX) kept whole
  kResid24 = 2,        // S_2:4 applied in the pass
  kResidDense = 3      // Q(dX) written whole; a global selection prunes it afterwards
};

// Row-wise quantization (blocks along columns) of a bf16 or f32 matrix.
void launch_quant_rows(int fmt, const void* x, bool in_f32, int64_t rows, int64_t cols,
                       int64_t ld, uint8_t* codes, void* scales, hipStream_t s);

// Column-wise quantization (blocks along rows), output transposed [cols][rows].
void launch_quant_cols(int fmt, const void* x, bool in_f32, int64_t rows, int64_t cols,
                       int64_t ld, uint8_t* codes, void* scales, hipStream_t s);

// Q(X), dX = X - Q(X), Q(dX), and S_2:4 / identity / none.  keep_mask and partials may be
// null.  partials (double [m][d/B]) receives the exact per-scale-block sums of squares of
// the dequantized Q(dX) (used by the block selection).
void launch_residual(int fmt, int mode, const uint16_t* X, int64_t m, int64_t d, int64_t ldx,
                     uint8_t* qx_codes, void* qx_scales, uint8_t* qr_codes, void* qr_scales,
                     uint8_t* keep_mask, double* partials, hipStream_t s);

// HiF4 K-major codes + metadata -> the split FP6 (E2M3) MFMA operand fragments.
// rows_pad (multiple of 32) rows are written; rows >= rows are zero.
void launch_pack_hif4(const uint8_t* codes, const uint32_t* meta, int64_t rows,
                      int64_t rows_pad, int64_t K, uint8_t* frag, uint8_t* frag_c1,
                      hipStream_t s);

// Global selections for the channel, block and unstructured 50% residual patterns.
// They read the dense Q(dX) (codes + scales), choose the kept set, then zero the pruned
// codes in place and write the element keep mask (and the channel/block mask).
struct SelectWs {
  double* keys;       // channel or block keys
  uint32_t* hist;     // radix-select histograms / counters
  uint32_t* state;    // selection state (prefix, counts)
  uint8_t* group_bits;  // kept channels / blocks (bit mask)
  uint32_t* tie_counts;  // per-workgroup tie counts (unstructured)
};
size_t select_ws_bytes(int sparsity, int fmt, int64_t m, int64_t d);
void carve_select_ws(void* base, int sparsity, int fmt, int64_t m, int64_t d, SelectWs& ws);
void launch_select(int fmt, int sparsity, int64_t m, int64_t d, uint8_t* qr_codes,
                   const void* qr_scales, const double* partials, uint8_t* keep_mask,
                   uint8_t* group_mask, const SelectWs& ws, hipStream_t s);

// FP4 GEMM  Y[M][N] = sum_t A_t[M][K] B[N][K]^T  with A_t = Q(X) and optionally S(Q(dX)).
struct GemmOperands {
  int fmt;
  int64_t M, N, K;
  // MXFP4: K-major codes + E8M0 scales of the A terms (row stride K/2 bytes)
  const uint8_t* a_codes[2];
  const uint8_t* a_scales[2];
  // HiF4: packed split fragments of the A terms and their level-1 codes
  const uint8_t* a_frag[2];
  const uint8_t* a_c1[2];
  int n_terms;               // 1 (Eq. 1) or 2 (with the residual term)
  const uint8_t* blockmask;  // optional: residual kept-block bits, (ceil(M/32), K/64) row-major
  // B: K-major codes + scales of Q(W) (row stride K/2 bytes)
  const uint8_t* b_codes;
  const void* b_scales;
  float* Y;
  int64_t ldy;
};
void launch_gemm(const GemmOperands& op, hipStream_t s);

}  // namespace resq
