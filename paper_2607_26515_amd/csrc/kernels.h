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
  kResidDense = 3,     // Q(dX) written whole; a global selection prunes it afterwards
  kResidNM8 = 4,       // S_k:8 applied in the pass (k = nm_keep)
  kResidNM4 = 5        // S_k:4 applied in the pass (k = nm_keep, k != 2)
};

// Row-wise quantization (blocks along columns) of a bf16 or f32 matrix.
void launch_quant_rows(int fmt, const void* x, bool in_f32, int64_t rows, int64_t cols,
                       int64_t ld, uint8_t* codes, void* scales, hipStream_t s);

// Column-wise quantization (blocks along rows) of a bf16 matrix written as fragment-major
// MFMA operands (pack.hip layout, PackMode `mode`): operand rows = the matrix's columns,
// operand K = its rows.  With rfrag (activation modes only), the same pass also writes the
// row-wise quantization (operand [rows][cols], blocks along cols) to rfrag / rfscale.
void launch_quant_cols_frag(int mode, const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                            uint8_t* frag, uint8_t* fscale, hipStream_t s, uint8_t* rfrag = nullptr,
                            uint8_t* rfscale = nullptr);

// Column-wise quantization (blocks along rows), output transposed [cols][rows].
void launch_quant_cols(int fmt, const void* x, bool in_f32, int64_t rows, int64_t cols,
                       int64_t ld, uint8_t* codes, void* scales, hipStream_t s);

// A producer fused into the forward's activation pass: instead of reading X, the pass forms
// X from the producer's inputs.  kProdSwiglu: X = silu(G) * U (the SwiGLU feeding a down
// projection) from G = g and U = u (m x d, row strides ldg and ldu, bf16 or float32), each
// element the bf16 nearest to its float64 value.  kProdRmsnorm: X = RMSNorm(H) * gamma from
// H = g (bf16, row stride ldg), gamma = u (d bf16 values) and rinv (m float32 factors
// 1 / sqrt(mean(H^2) + eps), written by launch_rms_rows), each element
// bf16(f32(f32(H r) gamma)).
enum ProducerKind { kProdSwiglu = 1, kProdRmsnorm = 2 };
struct Producer {
  const void* g;
  const void* u;
  int64_t ldg, ldu;
  bool f32;
  int kind;
  const float* rinv;
};

// The RMSNorm producer's per-row factors: rinv[i] = f32(1 / f32(sqrt(f32(f32(s_i / d) + eps))))
// with s_i the float32 nearest to the exact sum of the squares of row i of H (bf16, m x d, row
// stride ldh), every float32 step rounded to nearest even.  d <= 2^18; eps >= 2^-126, finite.
constexpr int64_t kRmsMaxD = (int64_t)1 << 18;
void launch_rms_rows(const uint16_t* H, int64_t m, int64_t d, int64_t ldh, float eps, float* rinv,
                     hipStream_t s);

// Q(X), dX = X - Q(X), Q(dX), and S_k:4 / S_k:8 (k = nm_keep) / identity / none.  keep_mask
// and partials may be null.  prod (frag = true only): X comes from that producer.  partials (double [m][d/B]) receives the exact per-scale-block sums of squares of
// the dequantized Q(dX) (used by the block selection).  frag = true writes MFMA fragments
// (pack.hip layout; codes -> fragment records, scales -> per-lane scale bytes) instead of
// K-major codes + scales: for both Q(X) and Q(dX) with the local kinds; with kResidDense
// Q(X) as fragments and Q(dX) K-major (qr_codes, qr_scales) for the selection that follows,
// and, with ehist (the element-wise selection's histogram, cleared beforehand by
// launch_select_clear), the exponent histogram of |Q(dX)|; with bkeys (frag and kResidDense,
// d % 64 == 0) the keys of the 32 x 64 blocks, summed as the block selection defines them
// (ceil(m / 32) x d / 64 doubles, block (I, J) at I * d / 64 + J).  keep_mask is ignored when
// frag is set.
void launch_residual(int fmt, int mode, const uint16_t* X, int64_t m, int64_t d, int64_t ldx,
                     uint8_t* qx_codes, void* qx_scales, uint8_t* qr_codes, void* qr_scales,
                     uint8_t* keep_mask, double* partials, hipStream_t s, bool frag = false,
                     uint32_t* ehist = nullptr, int nm_keep = 2, const Producer* prod = nullptr,
                     double* bkeys = nullptr);

// MFMA operand packing (pack.hip): K-major codes + scales -> fragment-major operands.
enum PackMode { kPackMx = 0, kPackHiA = 1, kPackHiB = 2 };
size_t frag_bytes(int mode, int64_t rows, int64_t K);
size_t frag_scale_bytes(int64_t rows, int64_t K);
// mask: 0 none; 1 kept channels, 2 kept 32 x 64 blocks (bit masks in gbits, as the channel
// and block selections write them): pruned elements are packed as the +0 code.
void launch_pack(int mode, const uint8_t* codes, const void* scales, int64_t rows, int64_t K,
                 uint8_t* frag, uint8_t* fscale, hipStream_t s, int mask = 0,
                 const uint8_t* gbits = nullptr);

// Global selections for the channel, block and element-wise residual patterns (sparsity
// 3, 4, 5).  They read the dense Q(dX) (codes + scales), keep the `keep` largest channels,
// blocks or elements, then zero the pruned codes in place and write the element keep mask
// (and the channel/block mask).
struct SelectWs {
  double* keys;       // channel or block keys
  uint32_t* hist;     // radix-select histograms / counters
  uint32_t* state;    // selection state (prefix, counts)
  uint8_t* group_bits;  // kept channels / blocks (bit mask)
  uint32_t* super_counts;  // [group of workgroups][64] tie counts (element-wise; cleared with hist)
  uint32_t* tie_counts;  // [workgroup][64] tie counts (element-wise)
};
size_t select_ws_bytes(int sparsity, int fmt, int64_t m, int64_t d);
int64_t select_max_items();  // most channels / blocks a channel or block selection ranks (2^31)
void carve_select_ws(void* base, int sparsity, int fmt, int64_t m, int64_t d, SelectWs& ws);
void launch_select(int fmt, int sparsity, int64_t m, int64_t d, int64_t keep, uint8_t* qr_codes,
                   const void* qr_scales, const double* partials, uint8_t* keep_mask,
                   uint8_t* group_mask, const SelectWs& ws, hipStream_t s);
// The same selections for the forward GEMM: S(Q(dX)) is written as fragment-major operand
// records (PackMode pack_mode) to frag / fscale; the K-major codes are left unpruned and no
// masks are written.  Block kind with partials = null: the residual pass has written the
// block keys to ws.keys.  For the element-wise kind the histogram (select_hist_words(m, d) words at
// ws.hist) must have been cleared (launch_select_clear) before the residual pass, which fills
// its exponent bins.
void launch_select_frag(int fmt, int sparsity, int64_t m, int64_t d, int64_t keep, uint8_t* qr_codes,
                        const void* qr_scales, const double* partials, const SelectWs& ws,
                        int pack_mode, uint8_t* frag, uint8_t* fscale, hipStream_t s);
int select_hist_words(int64_t m, int64_t d);  // words to clear at ws.hist (histograms, group counts)
// Clears the element-wise selection's histograms and group counts (ws.hist).
void launch_select_clear(const SelectWs& ws, int64_t m, int64_t d, hipStream_t s);

// FP4 GEMM  Y[M][N] = sum_t A_t[M][K] B[N][K]^T  with A_t = Q(X) and optionally S(Q(dX)),
// all operands fragment-major (pack.hip).  Operand A is one buffer holding the fragments and
// scale bytes of every term at the given byte offsets; operand B is one buffer holding its
// fragments and scale bytes.  Each buffer is below 4 GiB (32-bit offsets).
struct GemmOperands {
  int fmt;
  int64_t M, N, K;
  int n_terms;               // 1 (Eq. 1) or 2 (with the residual term)
  const uint8_t* a;
  size_t a_bytes;
  size_t a_frag_off[2], a_sc_off[2];
  const uint8_t* b;
  size_t b_bytes;
  size_t b_frag_off, b_sc_off;
  void* Y;                   // float32, or bf16 bits when out_bf16
  int64_t ldy;
  bool out_bf16;             // Y rounded to bf16 (nearest, ties to even) from float32
  // optional split-K scratch of gemm_split_scratch bytes (null: no K split)
  float* partial;
};
// Returns false (and launches nothing) when an operand buffer or offset does not fit the
// 32-bit offsets or an operand region lies outside its buffer.
bool launch_gemm(const GemmOperands& op, hipStream_t s);
// Scratch bytes a launch_gemm of this shape uses for its K split (0: it does not split).
size_t gemm_split_scratch(int fmt, int64_t M, int64_t N, int64_t K);
// The plan launch_gemm takes for these sizes: tile configuration (0: 64x64, 1: 128x256,
// 2: 128x192, 3: 128x192 in eight waves, 4: 64x128), K split, K groups and stages.
void gemm_plan_info(int fmt, int64_t M, int64_t N, int64_t K, bool may_split, int32_t info[4]);
// Whether launch_gemm handles these sizes: the A buffer of n_terms terms (fragments and
// scales, each 256-byte aligned) and the B buffer fit 32-bit offsets.
bool gemm_supported(int fmt, int64_t M, int64_t N, int64_t K, int n_terms);

// Mixed-precision GEMM (mixed.hip): Y[M][N] = A[M][K] B[N][K]^T in float32 on the bf16 MFMA.
// A is bf16 (row-major, row stride lda).  B is FP4 (K-major codes and scales of format fmt)
// when b_codes is not null, else bf16 rows (b_dense, row stride ldb).  A, b_codes and b_dense
// are 16-byte aligned with lda, ldb % 8 == 0, HiF4 scales 4-byte aligned, K a multiple of the
// format's block, and mixed_gemm_supported(K, lda, ldb, b_codes != null) holds.
void launch_mixed_gemm(int fmt, int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                       const uint8_t* b_codes, const void* b_scales, const uint16_t* b_dense, int64_t ldb,
                       float* Y, int64_t ldy, hipStream_t s);
// Whether one operand row of these strides fits the kernel's 32-bit buffer offsets (larger
// matrices are split over several launches).
bool mixed_gemm_supported(int64_t K, int64_t lda, int64_t ldb, bool b_quantized);
// Q(X) along rows (blocks along cols) written as its dequantized values in bf16 (exact): out
// is rows x cols with row stride ldo (8-byte aligned, ldo % 4 == 0).
void launch_quant_rows_bf16(int fmt, const uint16_t* x, int64_t rows, int64_t cols, int64_t ld, uint16_t* out,
                            int64_t ldo, hipStream_t s);

// p[0 .. n) = 0 (a fill kernel: callers may capture the library's launches in a graph).
void launch_zero_f32(float* p, int64_t n, hipStream_t s);

// Activation statistics (diag.hip): stats receives 9 doubles (see resq_diagnostics);
// partials is diag_ws_bytes(m, d) bytes of scratch.
size_t diag_ws_bytes(int64_t m, int64_t d);
void launch_diagnostics(int fmt, const uint16_t* X, int64_t m, int64_t d, int64_t ldx, float thr,
                        double* stats, double* partials, hipStream_t s);

}  // namespace resq
