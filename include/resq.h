/*
 * resq.h - C ABI of the Rollout-ResQ FP4 linear layer for AMD Instinct MI355X (gfx950).
 *
 * The layer is the rollout projection of "HiFloat4 Format for End-To-End Reinforcement
 * Learning Post-Training of Large Language Models" (Sec. 4.3, Eq. 4):
 *
 *     Y = Q(X) Q(W)^T + S(Q(dX)) Q(W)^T,   dX = X - Q(X)   (Eq. 2)
 *
 * with X (m x d, bf16 activations), W (n x d, bf16 weights), Q a block-scaled FP4
 * quantizer (MXFP4 or HiF4, Sec. 3) and S a sparsity function (Sec. 4.3).  S = none gives
 * the plain FP4 linear of Eq. 1, S = identity gives ResQ-Dense (Eq. 3).  The training
 * policy's FP4 backward GEMMs (Sec. 1, Sec. 4.1: forward and backward at 4 bits) are
 * provided by resq_linear_bwd.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers named x, X, W, dY, Y, dX, dW, codes, scales, masks and workspace are DEVICE
 *   pointers on the current HIP device; the caller owns every buffer.  The library
 *   allocates no device memory in these calls: scratch comes from `workspace`
 *   (size from resq_workspace_size), which must be 256-byte aligned.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).  Every call only
 *   enqueues work on that stream and returns; results are ready when the stream is.
 * - bf16 tensors are passed as uint16_t bit patterns; float outputs are IEEE float32.
 * - Matrices are row-major; `ld*` is the row stride in elements (>= the row length).
 * - Return value: RESQ_OK (0) or a negative resq_status.  Argument and shape errors are
 *   detected on the host before anything is enqueued; resq_last_error() then describes the
 *   problem (thread-local, valid until the next call on the same thread).  RESQ_ERR_HIP
 *   reports a failed launch (hipGetLastError after enqueueing).
 * - Inputs must be finite (no NaN / Inf); bf16 subnormals and signed zeros are handled.
 *
 * Quantized tensor layout ("K-major"): a tensor quantized in blocks along its contraction
 * axis K is stored as `outer` rows of K elements:
 *   codes : uint8 [outer][K/2]   two 4-bit codes per byte, element 2i in the low nibble;
 *                                a code is sign << 3 | magnitude.
 *   scales: MXFP4 -> uint8  [outer][K/32]  E8M0 code (exponent + 127) of each 32-block;
 *           HiF4  -> uint32 [outer][K/64]  bits 0-7: E6M2 level-1 scale code; bit 8+g:
 *                                level-2 bit of 8-element group g; bit 16+h: level-3 bit of
 *                                4-element group h (a set bit halves the scale above it).
 * MXFP4 element magnitudes: {0, .5, 1, 1.5, 2, 3, 4, 6} (E2M1); value = mag * 2^(E8M0-127).
 * HiF4 element magnitudes : k/4, k = 0..7 (S1P2); value = k/4 * s1 * 2^-(b2+b3) with
 *   s1 = 2^(c>>2 - 31) * (1 + (c&3)/4).  The paper fixes HiF4's three-level structure
 *   (Sec. 3) but not its group sizes, E6M2 bias or scale-selection rule; the library
 *   implements one stated reading (8- and 4-element groups, bias 31, smallest non-clipping
 *   scale at each level, round to nearest with ties to the even code).
 *
 * Bit masks: bit b of byte i is element 8i + b along a row.
 */
#ifndef RESQ_H
#define RESQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { RESQ_MXFP4 = 0, RESQ_HIF4 = 1 } resq_format;

/* Sparsity function S applied to the quantized residual Q(dX) (Sec. 4.3). */
typedef enum {
  RESQ_S_NONE = 0,          /* no residual term: plain FP4 linear, Eq. 1 */
  RESQ_S_IDENTITY = 1,      /* ResQ-Dense, Eq. 3 */
  RESQ_S_2_4 = 2,           /* S_2:4: keep the 2 largest |values| of every 4 along d */
  RESQ_S_CHANNEL50 = 3,     /* S_50%: keep the floor(d/2) channels (columns) of largest L2 norm */
  RESQ_S_BLOCK32X64_50 = 4, /* S^{32x64}_50%: keep half of the 32-row x 64-column blocks */
  RESQ_S_UNSTRUCT50 = 5     /* keep the floor(m*d/2) largest |values| of the tensor */
} resq_sparsity;

/*
 * Other levels and N:M patterns of the same sparsity functions.  Sec. 4.3 defines the
 * semi-structured pattern for any M:N and the channel and block patterns for any kept
 * fraction alpha; the paper evaluates 50% only and leaves other levels open (Sec. 6).  These
 * codes are accepted wherever a sparsity argument is:
 *   RESQ_S_NM(k, g)       keep the k largest |values| of every g consecutive elements along d;
 *                         g = 4 or 8, 1 <= k < g; d must be a multiple of g.
 *                         RESQ_S_NM(2, 4) computes exactly what RESQ_S_2_4 does.
 *   RESQ_S_CHANNEL(p)     keep the floor(d * p / 100) channels of largest L2 norm
 *   RESQ_S_BLOCK32X64(p)  keep floor(nblocks * p / 100) of the ceil(m/32) * (d/64) blocks
 *   RESQ_S_UNSTRUCT(p)    keep the floor(m * d * p / 100) largest |values|
 * with 1 <= p <= 99 (p = 50 is the matching RESQ_S_*50 kind).  Ranking, ties and limits are
 * those of the 50% kinds; a count that rounds down to 0 keeps nothing.  Any other value is
 * rejected with RESQ_ERR_ARG.
 */
#define RESQ_S_NM(k, g) (0x100 | ((k) << 4) | (g))
#define RESQ_S_CHANNEL(p) (0x200 | (p))
#define RESQ_S_BLOCK32X64(p) (0x300 | (p))
#define RESQ_S_UNSTRUCT(p) (0x400 | (p))

typedef enum {
  RESQ_OK = 0,
  RESQ_ERR_ARG = -1,         /* NULL pointer, bad enum, negative size, ld too small */
  RESQ_ERR_SHAPE = -2,       /* a blocked axis is not a multiple of the block size */
  RESQ_ERR_UNSUPPORTED = -3, /* valid but not implemented combination */
  RESQ_ERR_HIP = -4,         /* HIP launch or runtime failure */
  RESQ_ERR_WORKSPACE = -5    /* workspace missing, too small or misaligned */
} resq_status;

typedef enum { RESQ_IN_BF16 = 0, RESQ_IN_F32 = 1 } resq_dtype;

typedef enum {
  RESQ_OP_RESIDUAL_SPARSIFY = 0,
  RESQ_OP_LINEAR_FWD = 1,
  RESQ_OP_LINEAR_BWD = 2,
  RESQ_OP_LINEAR_FWD_PREPARED = 3,
  RESQ_OP_DIAGNOSTICS = 4,
  RESQ_OP_LINEAR_W16A4 = 5,
  RESQ_OP_LINEAR_FWD_RMSNORM = 6
} resq_op;

/*
 * resq_quantize - Q: block-scaled FP4 quantization of one matrix (Sec. 3).
 *
 * x      : rows x cols, bf16 (in_dtype = RESQ_IN_BF16) or float32 (RESQ_IN_F32), row stride
 *          ld elements.
 * axis   : 1 -> blocks run along cols (each row is quantized on its own); output layout
 *               [rows][cols] K-major with K = cols.  Requires cols % B == 0.
 *          0 -> blocks run along rows (each column is quantized on its own), as the
 *               backward GEMMs need ("transposed block scaling"); output layout
 *               [cols][rows] K-major with K = rows, i.e. the transpose.  Requires
 *               rows % B == 0.
 *          B = 32 (MXFP4) or 64 (HiF4).
 * codes  : output, uint8 [outer][K/2]; scales: output, see the layout above.
 * Rounding is to nearest, ties to the even code, saturating; the scale choice is the
 * format's (MXFP4: floor(log2 max|x|) - 2 clamped to [-127, 127]; HiF4: see above).
 */
int resq_quantize(int format, const void* x, int in_dtype, int64_t rows, int64_t cols,
                  int64_t ld, int axis, uint8_t* codes, void* scales, void* stream);

/*
 * resq_residual_sparsify - Q(X), dX = X - Q(X) (Eq. 2, formed in float32), Q(dX) with fresh
 * block scales, and S(Q(dX)) (Sec. 4.3), the activation side of Eq. 4.
 *
 * X         : m x d bf16, row stride ldx; d must be a multiple of 64 for HiF4, 32 for
 *             MXFP4, of 4 for S_2:4 (of g for RESQ_S_NM(k, g)) and of 64 for the block kinds.
 * qx_codes, qx_scales : output Q(X), layout [m][d] K-major.
 * qr_codes, qr_scales : output S(Q(dX)): pruned elements hold the +0 code, scales are those
 *             of Q(dX).  May be NULL when sparsity == RESQ_S_NONE.
 * keep_mask : output, uint8 [m][d/8], 1 = element kept by S (NULL to skip).
 * group_mask: output, kept channels (uint8 [d/8]) for the channel kinds, kept blocks
 *             (uint8 [ceil(ceil(m/32) * (d/64) / 8)], blocks row-major) for the
 *             32 x 64 block kinds; ignored otherwise (NULL allowed).
 * Ranking (channel, block, unstructured): by sum of squares of the dequantized Q(dX) values
 * (|value| for unstructured) in float64, ties to the lowest index; a channel's sum runs over
 * rows 0..m-1 in order; a block's over its rows in order, each row adding its per-scale-block
 * partial sums (exact) in column order.
 * Alignment: codes 16 bytes, keep_mask and HiF4 scales 4 bytes (RESQ_ERR_ARG otherwise).
 * Limits (RESQ_ERR_UNSUPPORTED beyond): channel kinds d <= 2^31; block kinds
 * ceil(m/32) * (d/64) <= 2^31 blocks; element-wise kinds m * d <= 2^31.
 * Workspace: resq_workspace_size(RESQ_OP_RESIDUAL_SPARSIFY, ...) bytes (0 for the local kinds).
 */
int resq_residual_sparsify(int format, int sparsity, const uint16_t* X, int64_t m, int64_t d,
                           int64_t ldx, uint8_t* qx_codes, void* qx_scales, uint8_t* qr_codes,
                           void* qr_scales, uint8_t* keep_mask, uint8_t* group_mask,
                           void* workspace, size_t workspace_bytes, void* stream);

/*
 * resq_linear_fwd - the rollout projection, Eq. 4 (Eq. 1 / Eq. 3 for S = none / identity):
 *     Y = Q(X) Q(W)^T + S(Q(X - Q(X))) Q(W)^T
 * X         : m x d bf16, row stride ldx (d as for resq_residual_sparsify).
 * qw_codes, qw_scales : Q(W) for W (n x d), from resq_quantize(W, axis = 1) in the same
 *             format; W is quantized once per policy update, not per call.
 * Y         : output, float32 m x n, row stride ldy >= n.  Products of FP4 values are exact;
 *             accumulation is float32.
 */
int resq_linear_fwd(int format, int sparsity, const uint16_t* X, int64_t m, int64_t d,
                    int64_t ldx, const uint8_t* qw_codes, const void* qw_scales, int64_t n,
                    float* Y, int64_t ldy, void* workspace, size_t workspace_bytes,
                    void* stream);

/*
 * resq_prepare_weights - lay Q(W) out as the GEMM's weight operand, once per policy update.
 * qw_codes, qw_scales : Q(W) from resq_quantize(W, axis = 1), W being n x d.
 * wprep     : output, device buffer of resq_prepared_weights_size(format, n, d) bytes,
 *             256-byte aligned.  The contents are an internal layout (the MFMA operand
 *             encoding of the same values: for MXFP4 the same E2M1/E8M0 codes, for HiF4 each
 *             element k 2^-b as a BF6 E3M2 code next to the block's level-1 scale code).
 * resq_linear_fwd_prepared is resq_linear_fwd with Q(W) given in this form; results are
 * identical.  Its workspace size is resq_workspace_size(RESQ_OP_LINEAR_FWD_PREPARED, ...).
 */
size_t resq_prepared_weights_size(int format, int64_t n, int64_t d);
int resq_prepare_weights(int format, const uint8_t* qw_codes, const void* qw_scales, int64_t n,
                         int64_t d, void* wprep, void* stream);
int resq_linear_fwd_prepared(int format, int sparsity, const uint16_t* X, int64_t m, int64_t d,
                             int64_t ldx, const void* wprep, int64_t n, float* Y, int64_t ldy,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * resq_linear_fwd_prepared_noalloc - resq_linear_fwd_prepared for callers that cannot
 * allocate device memory or hand the library a workspace (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  Same arguments without the
 * workspace, same kernels, same result bit for bit.  Its scratch (the MFMA operands of Q(X)
 * and S(Q(dX)), the selection's keys and counters, split-K partial tiles) is a static
 * device array of RESQ_NOALLOC_SCRATCH_BYTES in the library, one copy per GPU, held until
 * the process ends; the first call on a device looks up that device's copy.  The call
 * allocates nothing.  It runs on the current HIP device (`stream` must belong to it).
 * Calls whose scratch need (resq_workspace_size(RESQ_OP_LINEAR_FWD_PREPARED, ...)) exceeds
 * RESQ_NOALLOC_SCRATCH_BYTES return RESQ_ERR_UNSUPPORTED before enqueueing anything.
 * Every call on one GPU shares that GPU's array and leaves its contents behind (the kernels
 * clear what they count into): calls that can overlap on one GPU (other streams, other
 * threads) race on it and must be serialized by the caller.
 */
#define RESQ_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int resq_linear_fwd_prepared_noalloc(int format, int sparsity, const uint16_t* X, int64_t m,
                                     int64_t d, int64_t ldx, const void* wprep, int64_t n,
                                     float* Y, int64_t ldy, void* stream);

/*
 * resq_linear_fwd_prepared_bf16 - resq_linear_fwd_prepared with a bf16 output: Y is m x n
 * bf16 (bit patterns, row stride ldy >= n), each element the float32 result of Eq. 4 (as
 * resq_linear_fwd_prepared computes it) rounded to the nearest bf16, ties to even.  Halves
 * the output bytes, which dominate the decode shapes' HBM traffic after Q(W).  Arguments,
 * workspace (resq_workspace_size(RESQ_OP_LINEAR_FWD_PREPARED, ...)) and errors are those of
 * resq_linear_fwd_prepared.
 */
int resq_linear_fwd_prepared_bf16(int format, int sparsity, const uint16_t* X, int64_t m,
                                  int64_t d, int64_t ldx, const void* wprep, int64_t n,
                                  uint16_t* Y, int64_t ldy, void* workspace,
                                  size_t workspace_bytes, void* stream);

/*
 * resq_linear_fwd_prepared_swiglu - resq_linear_fwd_prepared for the down projection of a
 * SwiGLU MLP, with the activation formed inside the quantization pass instead of being read:
 *     X = silu(G) * U,   silu(g) = g / (1 + exp(-g)),
 * each element the bf16 nearest to the float64 value of silu(g) * u (ties to even), i.e. the
 * bf16 activation the unfused model hands to the linear, up to that one rounding.  X is never
 * written to memory: the pass reads G and U, forms X, then computes Q(X), dX, Q(dX) and S as
 * the other forward entry points do (Eq. 4).
 * G, U      : m x d, bf16 (in_dtype = RESQ_IN_BF16) or float32 (RESQ_IN_F32), row strides
 *             ldg, ldu >= d (for a gate/up projection output laid out [gate | up] with row
 *             stride 2d: G = base, U = base + d, ldg = ldu = 2d); element-size aligned.
 *             |silu(g) * u| must stay below the largest bf16 (3.39e38).
 * wprep, n, Y, ldy, workspace (resq_workspace_size(RESQ_OP_LINEAR_FWD_PREPARED, ...)) and
 * errors: as resq_linear_fwd_prepared; Y is float32.
 */
int resq_linear_fwd_prepared_swiglu(int format, int sparsity, const void* G, const void* U,
                                    int in_dtype, int64_t m, int64_t d, int64_t ldg, int64_t ldu,
                                    const void* wprep, int64_t n, float* Y, int64_t ldy,
                                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * resq_linear_fwd_prepared_rmsnorm - resq_linear_fwd_prepared for a projection that takes an
 * RMSNorm output (the qkv and gate/up projections of the Qwen2.5 models of Sec. 5.1), with the
 * normalization formed inside the quantization pass instead of being read:
 *     X = RMSNorm(H) * gamma,   per row: s = f32(sum_j H_j^2) (the exact sum, rounded once),
 *     r = f32(1 / f32(sqrt(f32(f32(s / d) + eps)))),   X_j = bf16(f32(f32(H_j r) gamma_j)),
 * every float32 step rounded to nearest even.  The exact sum makes X independent of summation
 * order: it is bit for bit the X of that definition.  A first launch computes r per row
 * (into the workspace); the activation pass reads H and gamma, forms X, then computes Q(X),
 * dX, Q(dX) and S as the other forward entry points do (Eq. 4).  X is never written.
 * H      : m x d bf16 (bit patterns), row stride ldh >= d, 2-byte aligned (16-byte aligned
 *          with ldh % 8 == 0 for 16-byte loads).  d <= 2^18 (else RESQ_ERR_UNSUPPORTED).
 * gamma  : d bf16 values.
 * eps    : finite, >= 2^-126 (else RESQ_ERR_ARG).
 * wprep, n, Y (float32), ldy and errors: as resq_linear_fwd_prepared.  Workspace:
 * resq_workspace_size(RESQ_OP_LINEAR_FWD_RMSNORM, format, sparsity, m, d, n) bytes.
 */
int resq_linear_fwd_prepared_rmsnorm(int format, int sparsity, const uint16_t* H, int64_t m,
                                     int64_t d, int64_t ldh, const uint16_t* gamma, float eps,
                                     const void* wprep, int64_t n, float* Y, int64_t ldy,
                                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * resq_linear_bwd - the FP4 training-policy backward GEMMs of the linear Y = X W^T:
 *     dX = Q_n(dY) Q_n(W)          (m x d, contraction over n)
 *     dW = Q_m(dY)^T Q_m(X)        (n x d, contraction over m)
 * where Q_a quantizes in blocks along axis a (each GEMM's contraction axis); no residual
 * term (ResQ is applied to the rollout only).
 * dY : m x n bf16, X : m x d bf16, W : n x d bf16, all contiguous (row stride = row length).
 * n must be a multiple of the block size (for dX) and m as well (for dW).
 * dX, dW : float32 outputs, contiguous; either may be NULL to skip that GEMM.  An empty
 *          contraction (n = 0 for dX, m = 0 for dW) writes zeros.
 */
int resq_linear_bwd(int format, const uint16_t* dY, const uint16_t* X, const uint16_t* W,
                    int64_t m, int64_t d, int64_t n, float* dX, float* dW, void* workspace,
                    size_t workspace_bytes, void* stream);

/*
 * resq_diagnostics - the activation statistics behind Figs. 2-4 (Sec. 4.2: zero values before
 * and after quantization, blocks holding outliers; Sec. 4.3: the error S_2:4 causes on Q(X)
 * and on Q(dX)) for one activation tensor X (m x d bf16, row stride ldx) and one format:
 *   stats[0] m * d                      stats[1] zeros of X (+0 or -0)
 *   stats[2] zeros of Q(X) (dequantized value 0, either sign)
 *   stats[3] quantization blocks, m * d / B (B = 32 MXFP4, 64 HiF4)
 *   stats[4] blocks holding some |x| > outlier_threshold (compared in float32; the paper
 *            does not define an outlier, so the threshold is the caller's)
 *   stats[5] sum of Q(X)^2              stats[6] sum of the squares S_2:4 prunes from Q(X)
 *   stats[7] sum of Q(dX)^2             stats[8] sum of the squares S_2:4 prunes from Q(dX)
 * The MSE of S_2:4 on Q(X) is stats[6] / stats[0] (on Q(dX) stats[8] / stats[0]); the RMSE is
 * its square root.  S_2:4 is the function RESQ_S_2_4 applies.
 * stats     : output, device buffer of RESQ_DIAG_STATS doubles.  Counts are exact; the sums
 *             are float64 additions of exact squares in a fixed order (the same on every run).
 * d must be a multiple of B.  Workspace: resq_workspace_size(RESQ_OP_DIAGNOSTICS, format,
 * 0, m, d, 0) bytes (256-byte aligned).
 */
#define RESQ_DIAG_STATS 9
int resq_diagnostics(int format, const uint16_t* X, int64_t m, int64_t d, int64_t ldx,
                     float outlier_threshold, double* stats, void* workspace,
                     size_t workspace_bytes, void* stream);

/* Workspace bytes needed by `op` (a resq_op) for these arguments; 0 on bad arguments. */
size_t resq_workspace_size(int op, int format, int sparsity, int64_t m, int64_t d, int64_t n);

/*
 * Mixed-precision rollout linears of the precision ablation (Sec. 4.2, Table 1, the W4A16
 * and W16A4 rows): only one GEMM operand is FP4, the other stays bf16.  They measure the
 * mixed-precision alternatives against which the paper argues for full FP4 GEMMs (Sec. 1).
 *
 * resq_linear_w4a16 - weight-only FP4: Y = X Q(W)^T (m x n float32, row stride ldy >= n).
 *   X: m x d bf16, row stride ldx (ldx % 8 == 0, X 16-byte aligned).  Q(W): K-major codes
 *   (n x d/2, 16-byte aligned) and scales (MXFP4 uint8 n x d/32; HiF4 uint32 n x d/64), as
 *   resq_quantize writes them.  d must be a multiple of the format's block.  No workspace.
 * resq_linear_w16a4 - activation-only FP4: Y = Q(X) W^T with Q(X) quantized along d inside
 *   the call and W: n x d bf16, row stride ldw (ldw % 8 == 0, W 16-byte aligned).  Workspace:
 *   resq_workspace_size(RESQ_OP_LINEAR_W16A4, format, 0, m, d, n) bytes (Q(X) as its
 *   dequantized bf16 values, m x d), 256-byte aligned.
 * Both compute in float32 on the bf16 MFMA: every FP4 value is exact in bf16, so every
 * product is exact and only the accumulation rounds.  Errors as resq_linear_fwd.
 */
int resq_linear_w4a16(int format, const uint16_t* X, int64_t m, int64_t d, int64_t ldx,
                      const uint8_t* qw_codes, const void* qw_scales, int64_t n, float* Y,
                      int64_t ldy, void* stream);
int resq_linear_w16a4(int format, const uint16_t* X, int64_t m, int64_t d, int64_t ldx,
                      const uint16_t* W, int64_t ldw, int64_t n, float* Y, int64_t ldy,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * The GEMM plan a call of these sizes runs (host-side query; nothing is enqueued and no GPU
 * is needed).  The GEMM computes Y[M][N] = sum over K: the forward linear has M = m, N = n,
 * K = d and may split K (split_allowed = 1); the backward's dX GEMM has M = m, N = d, K = n,
 * and its dW GEMM M = n, N = d, K = m, neither split (split_allowed = 0).
 * info receives four values: [0] tile configuration (RESQ_TILE_*), [1] K split count,
 * [2] K groups per workgroup, [3] LDS pipeline stages.  Returns RESQ_ERR_ARG for an unknown
 * format, negative sizes or a NULL info.
 */
enum { RESQ_TILE_64x64 = 0, RESQ_TILE_128x256 = 1, RESQ_TILE_128x192 = 2, RESQ_TILE_128x192_8W = 3,
       RESQ_TILE_64x128 = 4 };
int resq_gemm_plan(int format, int64_t M, int64_t N, int64_t K, int split_allowed, int32_t info[4]);

/* Human-readable description of the last non-OK status on this thread ("" if none). */
const char* resq_last_error(void);

/* Library version string. */
const char* resq_version(void);

/*
 * Kernel timing (diagnostics; off by default).  While enabled, every kernel the library
 * enqueues is timed with two HIP events on the same stream (event objects are host-side
 * handles; no device memory is allocated).  The GEMMs ("gemm", with a K split's reduction),
 * the forward's activation pass ("residual" in the forward entry points) and "diagnostics"
 * carry the events in their kernel dispatches, so the interval is the kernels' execution as a
 * kernel trace measures it; the other families record them around the enqueue, which adds
 * the dispatch gap (a few microseconds).  resq_profile_read synchronizes the
 * recorded events and returns, for the kernel family `name` ("residual", "quant_rows",
 * "quant_cols", "pack_hif4", "select", "gemm", "diagnostics", "mixed"), the number of launches and their summed
 * duration in milliseconds since the last reset.  Returns RESQ_ERR_ARG for an unknown name.
 */
int resq_profile_enable(int on);
void resq_profile_reset(void);
int resq_profile_read(const char* name, int64_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* RESQ_H */
