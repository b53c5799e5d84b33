// C ABI of the ResQ FP4 linear layer (declared in include/resq.h): argument validation,
// workspace carving and kernel dispatch.  Nothing here allocates device memory.
#include "resq.h"

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <algorithm>
#include <cstdio>
#include <cmath>
#include <mutex>
#include <string>

#include "kernels.h"
#include "profiler.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return RESQ_OK;
}

int check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(RESQ_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

int64_t block_of(int fmt) { return fmt == RESQ_MXFP4 ? 32 : 64; }
size_t scale_bytes(int fmt, int64_t outer, int64_t K) {
  return fmt == RESQ_MXFP4 ? (size_t)(outer * (K / 32)) : (size_t)(outer * (K / 64)) * 4;
}
size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

bool valid_format(int f) { return f == RESQ_MXFP4 || f == RESQ_HIF4; }

// A decoded sparsity argument: the family (named by its 50% enum value: RESQ_S_2_4 stands
// for every k:g pattern, RESQ_S_CHANNEL50 / _BLOCK32X64_50 / _UNSTRUCT50 for every level of
// the global kinds) and its parameters.
struct Sp {
  int kind = -1;           // -1: not a valid sparsity code
  int keep = 2, group = 4;  // k:g patterns
  int pct = 50;             // global kinds: percent of the channels / blocks / elements kept
};

Sp decode_sparsity(int code) {
  Sp sp;
  if (code >= RESQ_S_NONE && code <= RESQ_S_UNSTRUCT50) {
    sp.kind = code;
    return sp;
  }
  const int family = code >> 8, low = code & 0xFF;
  if (family == 1) {
    const int k = low >> 4, g = low & 15;
    if ((g == 4 || g == 8) && k >= 1 && k < g) {
      sp.kind = RESQ_S_2_4;
      sp.keep = k;
      sp.group = g;
    }
  } else if (family >= 2 && family <= 4 && low >= 1 && low <= 99) {
    sp.kind = family == 2 ? RESQ_S_CHANNEL50 : family == 3 ? RESQ_S_BLOCK32X64_50 : RESQ_S_UNSTRUCT50;
    sp.pct = low;
  }
  return sp;
}

bool global_kind(const Sp& sp) {
  return sp.kind == RESQ_S_CHANNEL50 || sp.kind == RESQ_S_BLOCK32X64_50 || sp.kind == RESQ_S_UNSTRUCT50;
}

// Items a global selection keeps: floor(count * pct / 100).
int64_t keep_count(const Sp& sp, int64_t m, int64_t d) {
  const int64_t count = sp.kind == RESQ_S_CHANNEL50 ? d
                        : sp.kind == RESQ_S_BLOCK32X64_50 ? ((m + 31) / 32) * (d / 64)
                                                          : m * d;
  return count * sp.pct / 100;
}

int resid_mode(const Sp& sp) {
  switch (sp.kind) {
    case RESQ_S_NONE: return resq::kResidNone;
    case RESQ_S_IDENTITY: return resq::kResidIdentity;
    case RESQ_S_2_4:
      return sp.group == 8 ? resq::kResidNM8 : sp.keep == 2 ? resq::kResid24 : resq::kResidNM4;
    default: return resq::kResidDense;
  }
}

// Sequential carving of one workspace block.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base((char*)b) {}
  void* take(size_t bytes) {
    void* p = base ? base + off : nullptr;
    off += align256(bytes);
    return p;
  }
};

// Activation-side buffers used by resq_linear_fwd and the selection.
struct ActWs {
  uint8_t* qr_codes;  // dense K-major Q(dX) (global selections only)
  void* qr_scales;
  uint8_t* frag_x;
  uint8_t* fsc_x;
  uint8_t* frag_r;
  uint8_t* fsc_r;
  float* gemm_partial;       // split-K partial tiles
  float* rinv;               // the RMSNorm producer's per-row factors
  resq::SelectWs sel;
};

int a_pack_mode(int fmt) { return fmt == RESQ_MXFP4 ? resq::kPackMx : resq::kPackHiA; }
int b_pack_mode(int fmt) { return fmt == RESQ_MXFP4 ? resq::kPackMx : resq::kPackHiB; }

// GEMM operands from fragment / scale arrays: every array of A lies at or after a_frag[0]
// (its buffer starts there), every array of B at or after b_frag.  launch_gemm rejects
// offsets outside the buffers.
resq::GemmOperands gemm_operands(int fmt, int64_t M, int64_t N, int64_t K, int n_terms,
                                 const uint8_t* const a_frag[2], const uint8_t* const a_sc[2],
                                 const uint8_t* b_frag, const uint8_t* b_sc, void* Y, int64_t ldy,
                                 bool out_bf16 = false) {
  resq::GemmOperands op{};
  op.fmt = fmt;
  op.M = M; op.N = N; op.K = K;
  op.n_terms = n_terms;
  const size_t af = resq::frag_bytes(a_pack_mode(fmt), M, K), bf = resq::frag_bytes(b_pack_mode(fmt), N, K);
  const size_t as = resq::frag_scale_bytes(M, K), bs = resq::frag_scale_bytes(N, K);
  op.a = a_frag[0];
  for (int t = 0; t < n_terms; ++t) {
    op.a_frag_off[t] = (size_t)(a_frag[t] - op.a);
    op.a_sc_off[t] = (size_t)(a_sc[t] - op.a);
    op.a_bytes = std::max(op.a_bytes, std::max(op.a_frag_off[t] + af, op.a_sc_off[t] + as));
  }
  op.b = b_frag;
  op.b_frag_off = 0;
  op.b_sc_off = (size_t)(b_sc - b_frag);
  op.b_bytes = std::max(bf, op.b_sc_off + bs);
  op.Y = Y; op.ldy = ldy; op.out_bf16 = out_bf16;
  return op;
}

// partials: the block kind's per-row scale-block sums (resq_residual_sparsify; the forward's
// residual pass writes the block keys instead and passes null).
size_t carve_select(Carver& c, int fmt, const Sp& sp, int64_t m, int64_t d, double** partials,
                    resq::SelectWs* sel) {
  const size_t start = c.off;
  void* part = (partials && sp.kind == RESQ_S_BLOCK32X64_50) ? c.take((size_t)m * (d / block_of(fmt)) * 8)
                                                             : nullptr;
  if (partials) *partials = (double*)part;
  const size_t sb = global_kind(sp) ? resq::select_ws_bytes(sp.kind, fmt, m, d) : 0;
  void* sw = sb ? c.take(sb) : nullptr;
  if (sel) {
    *sel = resq::SelectWs{};
    if (sw) resq::carve_select_ws(sw, sp.kind, fmt, m, d, *sel);
  }
  return c.off - start;
}

// Prepared weights: fragment-major codes, then one scale byte per lane record.
size_t prepared_bytes(int fmt, int64_t n, int64_t d) {
  return align256(resq::frag_bytes(b_pack_mode(fmt), n, d)) + align256(resq::frag_scale_bytes(n, d));
}

void carve_prepared(const void* base, int fmt, int64_t n, int64_t d, const uint8_t** frag,
                    const uint8_t** fsc) {
  const uint8_t* b = (const uint8_t*)base;
  *frag = b;
  *fsc = b + align256(resq::frag_bytes(b_pack_mode(fmt), n, d));
}

size_t carve_fwd(void* base, int fmt, const Sp& sp, int64_t m, int64_t d, int64_t n, ActWs* w,
                 bool rms = false) {
  Carver c(base);
  ActWs t{};
  if (global_kind(sp)) {  // the dense K-major Q(dX) the selection ranks
    t.qr_codes = (uint8_t*)c.take((size_t)m * d / 2);
    t.qr_scales = c.take(scale_bytes(fmt, m, d));
  }
  carve_select(c, fmt, sp, m, d, nullptr, &t.sel);
  t.frag_x = (uint8_t*)c.take(resq::frag_bytes(a_pack_mode(fmt), m, d));
  t.fsc_x = (uint8_t*)c.take(resq::frag_scale_bytes(m, d));
  if (sp.kind != RESQ_S_NONE) {
    t.frag_r = (uint8_t*)c.take(resq::frag_bytes(a_pack_mode(fmt), m, d));
    t.fsc_r = (uint8_t*)c.take(resq::frag_scale_bytes(m, d));
  }
  const size_t pb = resq::gemm_split_scratch(fmt, m, n, d);
  if (pb > 0) t.gemm_partial = (float*)c.take(pb);
  if (rms) t.rinv = (float*)c.take((size_t)m * sizeof(float));
  if (w) *w = t;
  return c.off;
}

struct BwdWs {
  uint8_t *fa, *fa_sc, *fb, *fb_sc;
  uint8_t *fr, *fr_sc;  // Q_n(dY) for dX when both gradients are computed (one pass over dY)
};

// The backward's GEMM operands, written fragment-major straight from bf16 dY, W and X and
// reused by the two GEMMs (the stream orders them).
size_t carve_bwd(void* base, int fmt, int64_t m, int64_t d, int64_t n, BwdWs* w) {
  Carver c(base);
  BwdWs t{};
  const size_t fa = std::max(resq::frag_bytes(a_pack_mode(fmt), m, n), resq::frag_bytes(a_pack_mode(fmt), n, m));
  const size_t fas = std::max(resq::frag_scale_bytes(m, n), resq::frag_scale_bytes(n, m));
  const size_t fb = std::max(resq::frag_bytes(b_pack_mode(fmt), d, n), resq::frag_bytes(b_pack_mode(fmt), d, m));
  const size_t fbs = std::max(resq::frag_scale_bytes(d, n), resq::frag_scale_bytes(d, m));
  t.fa = (uint8_t*)c.take(fa);
  t.fa_sc = (uint8_t*)c.take(fas);
  t.fb = (uint8_t*)c.take(fb);
  t.fb_sc = (uint8_t*)c.take(fbs);
  t.fr = (uint8_t*)c.take(resq::frag_bytes(a_pack_mode(fmt), m, n));
  t.fr_sc = (uint8_t*)c.take(resq::frag_scale_bytes(m, n));
  if (w) *w = t;
  return c.off;
}

int check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return ok();
  if (ws == nullptr) return fail(RESQ_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", need);
  if ((uintptr_t)ws % 256 != 0) return fail(RESQ_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (have < need) return fail(RESQ_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  return ok();
}

int check_activation_args(int format, int sparsity, const Sp& sp, const void* X, int64_t m,
                          int64_t d, int64_t ldx) {
  if (!valid_format(format)) return fail(RESQ_ERR_ARG, "unknown format %d", format);
  if (sp.kind < 0) return fail(RESQ_ERR_ARG, "unknown sparsity %d", sparsity);
  if (m < 0 || d < 0) return fail(RESQ_ERR_ARG, "negative size (m=%lld, d=%lld)", (long long)m, (long long)d);
  if (ldx < d) return fail(RESQ_ERR_ARG, "ldx (%lld) < d (%lld)", (long long)ldx, (long long)d);
  if (d % block_of(format) != 0)
    return fail(RESQ_ERR_SHAPE, "d (%lld) is not a multiple of the block size %lld", (long long)d, (long long)block_of(format));
  if (sp.kind == RESQ_S_2_4 && d % sp.group != 0)
    return fail(RESQ_ERR_SHAPE, "%d:%d sparsity needs d %% %d == 0 (d=%lld)", sp.keep, sp.group, sp.group, (long long)d);
  if (sp.kind == RESQ_S_BLOCK32X64_50 && d % 64 != 0)
    return fail(RESQ_ERR_SHAPE, "32x64 block sparsity needs d %% 64 == 0 (d=%lld)", (long long)d);
  if (sp.kind == RESQ_S_CHANNEL50 && d > resq::select_max_items())
    return fail(RESQ_ERR_UNSUPPORTED, "channel selection supports d <= %lld (d=%lld)",
                (long long)resq::select_max_items(), (long long)d);
  if (sp.kind == RESQ_S_BLOCK32X64_50 && ((m + 31) / 32) * (d / 64) > resq::select_max_items())
    return fail(RESQ_ERR_UNSUPPORTED, "block selection supports ceil(m/32)*(d/64) <= %lld blocks",
                (long long)resq::select_max_items());
  if (sp.kind == RESQ_S_UNSTRUCT50 && m * d > ((int64_t)1 << 31))
    return fail(RESQ_ERR_UNSUPPORTED, "element-wise selection supports m*d <= 2^31 (m*d=%lld)", (long long)(m * d));
  if (m > 0 && d > 0 && X == nullptr) return fail(RESQ_ERR_ARG, "X is NULL");
  return ok();
}

int run_activation_side(int format, const Sp& sp, const uint16_t* X, int64_t m, int64_t d,
                        int64_t ldx, uint8_t* qx_codes, void* qx_scales, uint8_t* qr_codes,
                        void* qr_scales, uint8_t* keep_mask, uint8_t* group_mask,
                        double* partials, const resq::SelectWs& sel, hipStream_t s) {
  {
    resq::ProfScope prof_(resq::kProfResidual, s);
    resq::launch_residual(format, resid_mode(sp), X, m, d, ldx, qx_codes, qx_scales, qr_codes,
                          qr_scales, keep_mask, partials, s, false, nullptr, sp.keep);
  }
  if (global_kind(sp)) {
    resq::ProfScope prof_(resq::kProfSelect, s);
    resq::launch_select(format, sp.kind, m, d, keep_count(sp, m, d), qr_codes, qr_scales, partials,
                        keep_mask, group_mask, sel, s);
  }
  return check_launch("residual/sparsify");
}

}  // namespace

extern "C" {

const char* resq_last_error(void) { return g_err.c_str(); }

const char* resq_version(void) { return "resq-gfx950 0.2"; }

int resq_gemm_plan(int format, int64_t M, int64_t N, int64_t K, int split_allowed, int32_t info[4]) {
  if (!valid_format(format)) return fail(RESQ_ERR_ARG, "unknown format %d", format);
  if (M < 0 || N < 0 || K < 0) return fail(RESQ_ERR_ARG, "negative size");
  if (!info) return fail(RESQ_ERR_ARG, "info is NULL");
  resq::gemm_plan_info(format, M, N, K, split_allowed != 0, info);
  return ok();
}

int resq_quantize(int format, const void* x, int in_dtype, int64_t rows, int64_t cols,
                  int64_t ld, int axis, uint8_t* codes, void* scales, void* stream) {
  if (!valid_format(format)) return fail(RESQ_ERR_ARG, "unknown format %d", format);
  if (in_dtype != RESQ_IN_BF16 && in_dtype != RESQ_IN_F32) return fail(RESQ_ERR_ARG, "unknown input dtype %d", in_dtype);
  if (axis != 0 && axis != 1) return fail(RESQ_ERR_ARG, "axis must be 0 or 1 (got %d)", axis);
  if (rows < 0 || cols < 0) return fail(RESQ_ERR_ARG, "negative size");
  if (ld < cols) return fail(RESQ_ERR_ARG, "ld (%lld) < cols (%lld)", (long long)ld, (long long)cols);
  const int64_t K = axis == 1 ? cols : rows;
  if (K % block_of(format) != 0)
    return fail(RESQ_ERR_SHAPE, "blocked axis length %lld is not a multiple of %lld", (long long)K, (long long)block_of(format));
  if (rows == 0 || cols == 0) return ok();
  if (!x || !codes || !scales) return fail(RESQ_ERR_ARG, "NULL pointer argument");
  hipStream_t s = (hipStream_t)stream;
  if (axis == 1)
    {
      resq::ProfScope prof_(resq::kProfQuantRows, s);
      resq::launch_quant_rows(format, x, in_dtype == RESQ_IN_F32, rows, cols, ld, codes, scales, s);
    }
  else
    {
      resq::ProfScope prof_(resq::kProfQuantCols, s);
      resq::launch_quant_cols(format, x, in_dtype == RESQ_IN_F32, rows, cols, ld, codes, scales, s);
    }
  return check_launch("resq_quantize");
}

size_t resq_workspace_size(int op, int format, int sparsity, int64_t m, int64_t d, int64_t n) {
  const Sp sp = decode_sparsity(sparsity);
  if (!valid_format(format) || sp.kind < 0 || m < 0 || d < 0 || n < 0) return 0;
  switch (op) {
    case RESQ_OP_RESIDUAL_SPARSIFY: {
      Carver c(nullptr);
      double* partials = nullptr;  // counted: this entry point writes the block partials
      carve_select(c, format, sp, m, d, &partials, nullptr);
      return c.off;
    }
    case RESQ_OP_LINEAR_FWD:
      return carve_fwd(nullptr, format, sp, m, d, n, nullptr) + prepared_bytes(format, n, d);
    case RESQ_OP_LINEAR_FWD_PREPARED: return carve_fwd(nullptr, format, sp, m, d, n, nullptr);
    case RESQ_OP_LINEAR_FWD_RMSNORM: return carve_fwd(nullptr, format, sp, m, d, n, nullptr, true);
    case RESQ_OP_LINEAR_BWD: return carve_bwd(nullptr, format, m, d, n, nullptr);
    case RESQ_OP_DIAGNOSTICS: return resq::diag_ws_bytes(m, d);
    case RESQ_OP_LINEAR_W16A4:
      return d % block_of(format) ? 0 : align256((size_t)m * d * 2);
    default: return 0;
  }
}

int resq_residual_sparsify(int format, int sparsity, const uint16_t* X, int64_t m, int64_t d,
                           int64_t ldx, uint8_t* qx_codes, void* qx_scales, uint8_t* qr_codes,
                           void* qr_scales, uint8_t* keep_mask, uint8_t* group_mask,
                           void* workspace, size_t workspace_bytes, void* stream) {
  const Sp sp = decode_sparsity(sparsity);
  int rc = check_activation_args(format, sparsity, sp, X, m, d, ldx);
  if (rc != RESQ_OK) return rc;
  if (m == 0 || d == 0) return ok();
  if (!qx_codes || !qx_scales) return fail(RESQ_ERR_ARG, "qx_codes / qx_scales is NULL");
  if (sp.kind != RESQ_S_NONE && (!qr_codes || !qr_scales))
    return fail(RESQ_ERR_ARG, "qr_codes / qr_scales is NULL");
  if ((uintptr_t)qx_codes % 16 || (uintptr_t)qr_codes % 16 || (uintptr_t)keep_mask % 4 ||
      (format == RESQ_HIF4 && ((uintptr_t)qx_scales % 4 || (uintptr_t)qr_scales % 4)))
    return fail(RESQ_ERR_ARG, "codes must be 16-byte, keep_mask and HiF4 scales 4-byte aligned");
  Carver c(workspace);
  double* partials = nullptr;
  resq::SelectWs sel{};
  carve_select(c, format, sp, m, d, &partials, &sel);
  rc = check_ws(workspace, workspace_bytes, c.off);
  if (rc != RESQ_OK) return rc;
  return run_activation_side(format, sp, X, m, d, ldx, qx_codes, qx_scales, qr_codes,
                             qr_scales, keep_mask, group_mask, partials, sel,
                             (hipStream_t)stream);
}

size_t resq_prepared_weights_size(int format, int64_t n, int64_t d) {
  if (!valid_format(format) || n < 0 || d < 0 || d % block_of(format) != 0) return 0;
  return prepared_bytes(format, n, d);
}

int resq_prepare_weights(int format, const uint8_t* qw_codes, const void* qw_scales, int64_t n,
                         int64_t d, void* wprep, void* stream) {
  if (!valid_format(format)) return fail(RESQ_ERR_ARG, "unknown format %d", format);
  if (n < 0 || d < 0) return fail(RESQ_ERR_ARG, "negative size");
  if (d % block_of(format) != 0)
    return fail(RESQ_ERR_SHAPE, "d (%lld) is not a multiple of the block size %lld", (long long)d, (long long)block_of(format));
  if (n == 0 || d == 0) return ok();
  if (!qw_codes || !qw_scales || !wprep) return fail(RESQ_ERR_ARG, "NULL pointer argument");
  if ((uintptr_t)qw_codes % 16 != 0 || (uintptr_t)wprep % 256 != 0 ||
      (format == RESQ_HIF4 && (uintptr_t)qw_scales % 4 != 0))
    return fail(RESQ_ERR_ARG, "qw_codes must be 16-byte and wprep 256-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  const uint8_t *frag, *fsc;
  carve_prepared(wprep, format, n, d, &frag, &fsc);
  {
    resq::ProfScope prof_(resq::kProfPack, s);
    resq::launch_pack(b_pack_mode(format), qw_codes, qw_scales, n, d, (uint8_t*)frag, (uint8_t*)fsc, s);
  }
  return check_launch("resq_prepare_weights");
}

namespace {

int linear_fwd_core(int format, const Sp& sp, const uint16_t* X, int64_t m, int64_t d,
                    int64_t ldx, const void* wprep, int64_t n, void* Y, int64_t ldy, bool out_bf16,
                    const ActWs& w, hipStream_t s, const resq::Producer* prod = nullptr) {
  if (global_kind(sp)) {
    // the residual pass writes Q(X) as MFMA fragments and the dense Q(dX) K-major (the
    // selection ranks all of it); the selection then writes S(Q(dX)) as fragments
    {
      resq::ProfScope prof_(resq::kProfResidual, s, true);
      const bool elem = sp.kind == RESQ_S_UNSTRUCT50;
      if (elem) resq::launch_select_clear(w.sel, m, d, s);  // the residual pass counts into it
      // the block kind: the pass writes the block keys, which the top-k then ranks directly
      const bool block = sp.kind == RESQ_S_BLOCK32X64_50;
      resq::launch_residual(format, resq::kResidDense, X, m, d, ldx, w.frag_x, w.fsc_x, w.qr_codes,
                            w.qr_scales, nullptr, nullptr, s, true, elem ? w.sel.hist : nullptr, 2, prod,
                            block ? w.sel.keys : nullptr);
    }
    resq::ProfScope prof_(resq::kProfSelect, s);
    resq::launch_select_frag(format, sp.kind, m, d, keep_count(sp, m, d), w.qr_codes, w.qr_scales,
                             nullptr, w.sel, a_pack_mode(format), w.frag_r, w.fsc_r, s);
  } else {
    // local kinds: the residual pass writes the MFMA fragments directly
    resq::ProfScope prof_(resq::kProfResidual, s, true);
    resq::launch_residual(format, resid_mode(sp), X, m, d, ldx, w.frag_x, w.fsc_x, w.frag_r,
                          w.fsc_r, nullptr, nullptr, s, true, nullptr, sp.keep, prod);
  }
  const uint8_t* af[2] = {w.frag_x, w.frag_r};
  const uint8_t* asc[2] = {w.fsc_x, w.fsc_r};
  const uint8_t *bf, *bsc;
  carve_prepared(wprep, format, n, d, &bf, &bsc);
  resq::GemmOperands op = gemm_operands(format, m, n, d, sp.kind == RESQ_S_NONE ? 1 : 2, af, asc,
                                        bf, bsc, Y, ldy, out_bf16);
  op.partial = w.gemm_partial;
  {
    resq::ProfScope prof_(resq::kProfGemm, s, true);
    if (!resq::launch_gemm(op, s)) return fail(RESQ_ERR_UNSUPPORTED, "GEMM operand layout rejected");
  }
  return check_launch("resq_linear_fwd");
}

int check_fwd_args(int format, int sparsity, const Sp& sp, const uint16_t* X, int64_t m,
                   int64_t d, int64_t ldx, int64_t n, const void* Y, int64_t ldy) {
  int rc = check_activation_args(format, sparsity, sp, X, m, d, ldx);
  if (rc != RESQ_OK) return rc;
  if (n < 0) return fail(RESQ_ERR_ARG, "negative n");
  if (ldy < n) return fail(RESQ_ERR_ARG, "ldy (%lld) < n (%lld)", (long long)ldy, (long long)n);
  if (m > 0 && n > 0 && !Y) return fail(RESQ_ERR_ARG, "Y is NULL");
  if (!resq::gemm_supported(format, m, n, d, sp.kind == RESQ_S_NONE ? 1 : 2))
    return fail(RESQ_ERR_UNSUPPORTED, "GEMM operands too large for 32-bit offsets (m=%lld, d=%lld, n=%lld)",
                (long long)m, (long long)d, (long long)n);
  return ok();
}

int linear_fwd_prepared(int format, int sparsity, const uint16_t* X, int64_t m, int64_t d,
                        int64_t ldx, const void* wprep, int64_t n, void* Y, int64_t ldy, bool out_bf16,
                        void* workspace, size_t workspace_bytes, void* stream) {
  const Sp sp = decode_sparsity(sparsity);
  int rc = check_fwd_args(format, sparsity, sp, X, m, d, ldx, n, Y, ldy);
  if (rc != RESQ_OK) return rc;
  if (m == 0 || n == 0) return ok();
  if (d > 0 && !wprep) return fail(RESQ_ERR_ARG, "wprep is NULL");
  if ((uintptr_t)wprep % 256 != 0) return fail(RESQ_ERR_ARG, "wprep must be 256-byte aligned");
  ActWs w{};
  const size_t need = carve_fwd(workspace, format, sp, m, d, n, &w);
  rc = check_ws(workspace, workspace_bytes, need);
  if (rc != RESQ_OK) return rc;
  return linear_fwd_core(format, sp, X, m, d, ldx, wprep, n, Y, ldy, out_bf16, w,
                         (hipStream_t)stream);
}

}  // namespace

int resq_linear_fwd_prepared(int format, int sparsity, const uint16_t* X, int64_t m, int64_t d,
                             int64_t ldx, const void* wprep, int64_t n, float* Y, int64_t ldy,
                             void* workspace, size_t workspace_bytes, void* stream) {
  return linear_fwd_prepared(format, sparsity, X, m, d, ldx, wprep, n, Y, ldy, false, workspace,
                             workspace_bytes, stream);
}

namespace {

// Scratch of resq_linear_fwd_prepared_noalloc: one static device array per GPU.  Host code
// never uses the array's name as an address; it uses the device address looked up once per
// device with hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[RESQ_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int device_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(RESQ_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(RESQ_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(RESQ_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ok();
}

}  // namespace

int resq_linear_fwd_prepared_noalloc(int format, int sparsity, const uint16_t* X, int64_t m,
                                     int64_t d, int64_t ldx, const void* wprep, int64_t n,
                                     float* Y, int64_t ldy, void* stream) {
  const Sp sp = decode_sparsity(sparsity);
  int rc = check_fwd_args(format, sparsity, sp, X, m, d, ldx, n, Y, ldy);
  if (rc != RESQ_OK) return rc;
  if (m == 0 || n == 0) return ok();
  if (d > 0 && !wprep) return fail(RESQ_ERR_ARG, "wprep is NULL");
  if ((uintptr_t)wprep % 256 != 0) return fail(RESQ_ERR_ARG, "wprep must be 256-byte aligned");
  const size_t need = carve_fwd(nullptr, format, sp, m, d, n, nullptr);
  if (need > RESQ_NOALLOC_SCRATCH_BYTES)
    return fail(RESQ_ERR_UNSUPPORTED,
                "resq_linear_fwd_prepared_noalloc: these sizes need %zu bytes of scratch, the static "
                "buffer holds %zu (use resq_linear_fwd_prepared with a workspace)",
                need, (size_t)RESQ_NOALLOC_SCRATCH_BYTES);
  void* base = nullptr;
  rc = device_scratch(&base);
  if (rc != RESQ_OK) return rc;
  ActWs w{};
  carve_fwd(base, format, sp, m, d, n, &w);
  return linear_fwd_core(format, sp, X, m, d, ldx, wprep, n, Y, ldy, false, w, (hipStream_t)stream);
}

int resq_linear_fwd_prepared_bf16(int format, int sparsity, const uint16_t* X, int64_t m,
                                  int64_t d, int64_t ldx, const void* wprep, int64_t n,
                                  uint16_t* Y, int64_t ldy, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  return linear_fwd_prepared(format, sparsity, X, m, d, ldx, wprep, n, Y, ldy, true, workspace,
                             workspace_bytes, stream);
}

int resq_linear_fwd_prepared_swiglu(int format, int sparsity, const void* G, const void* U,
                                    int in_dtype, int64_t m, int64_t d, int64_t ldg, int64_t ldu,
                                    const void* wprep, int64_t n, float* Y, int64_t ldy,
                                    void* workspace, size_t workspace_bytes, void* stream) {
  const Sp sp = decode_sparsity(sparsity);
  if (in_dtype != RESQ_IN_BF16 && in_dtype != RESQ_IN_F32)
    return fail(RESQ_ERR_ARG, "unknown input dtype %d", in_dtype);
  int rc = check_fwd_args(format, sparsity, sp, (const uint16_t*)G, m, d, std::min(ldg, ldu), n, Y, ldy);
  if (rc != RESQ_OK) return rc;
  if (m > 0 && d > 0 && !U) return fail(RESQ_ERR_ARG, "U is NULL");
  if (m == 0 || n == 0) return ok();
  if (d > 0 && !wprep) return fail(RESQ_ERR_ARG, "wprep is NULL");
  if ((uintptr_t)wprep % 256 != 0) return fail(RESQ_ERR_ARG, "wprep must be 256-byte aligned");
  const size_t esz = in_dtype == RESQ_IN_F32 ? 4 : 2;
  if ((uintptr_t)G % esz != 0 || (uintptr_t)U % esz != 0)
    return fail(RESQ_ERR_ARG, "G and U must be aligned to their element size");
  ActWs w{};
  const size_t need = carve_fwd(workspace, format, sp, m, d, n, &w);
  rc = check_ws(workspace, workspace_bytes, need);
  if (rc != RESQ_OK) return rc;
  const resq::Producer prod{G, U, ldg, ldu, in_dtype == RESQ_IN_F32, resq::kProdSwiglu, nullptr};
  return linear_fwd_core(format, sp, nullptr, m, d, 0, wprep, n, Y, ldy, false, w,
                         (hipStream_t)stream, &prod);
}

int resq_linear_fwd_prepared_rmsnorm(int format, int sparsity, const uint16_t* H, int64_t m,
                                     int64_t d, int64_t ldh, const uint16_t* gamma, float eps,
                                     const void* wprep, int64_t n, float* Y, int64_t ldy,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  const Sp sp = decode_sparsity(sparsity);
  int rc = check_fwd_args(format, sparsity, sp, H, m, d, ldh, n, Y, ldy);
  if (rc != RESQ_OK) return rc;
  if (!std::isfinite(eps) || !(eps >= 0x1p-126f))
    return fail(RESQ_ERR_ARG, "eps (%g) must be finite and at least 2^-126", (double)eps);
  if (d > resq::kRmsMaxD)
    return fail(RESQ_ERR_UNSUPPORTED, "the RMSNorm producer supports d <= %lld (d=%lld)",
                (long long)resq::kRmsMaxD, (long long)d);
  if (m > 0 && d > 0 && !gamma) return fail(RESQ_ERR_ARG, "gamma is NULL");
  if (m == 0 || n == 0) return ok();
  if (d > 0 && !wprep) return fail(RESQ_ERR_ARG, "wprep is NULL");
  if ((uintptr_t)wprep % 256 != 0) return fail(RESQ_ERR_ARG, "wprep must be 256-byte aligned");
  if ((uintptr_t)H % 2 != 0 || (uintptr_t)gamma % 2 != 0)
    return fail(RESQ_ERR_ARG, "H and gamma must be 2-byte aligned");
  ActWs w{};
  const size_t need = carve_fwd(workspace, format, sp, m, d, n, &w, true);
  rc = check_ws(workspace, workspace_bytes, need);
  if (rc != RESQ_OK) return rc;
  const hipStream_t s = (hipStream_t)stream;
  {
    resq::ProfScope prof_(resq::kProfResidual, s, true);
    resq::launch_rms_rows(H, m, d, ldh, eps, w.rinv, s);
  }
  const resq::Producer prod{H, gamma, ldh, 0, false, resq::kProdRmsnorm, w.rinv};
  return linear_fwd_core(format, sp, nullptr, m, d, 0, wprep, n, Y, ldy, false, w, s, &prod);
}

int resq_linear_fwd(int format, int sparsity, const uint16_t* X, int64_t m, int64_t d,
                    int64_t ldx, const uint8_t* qw_codes, const void* qw_scales, int64_t n,
                    float* Y, int64_t ldy, void* workspace, size_t workspace_bytes,
                    void* stream) {
  const Sp sp = decode_sparsity(sparsity);
  int rc = check_fwd_args(format, sparsity, sp, X, m, d, ldx, n, Y, ldy);
  if (rc != RESQ_OK) return rc;
  if (m == 0 || n == 0) return ok();
  if (d > 0 && (!qw_codes || !qw_scales)) return fail(RESQ_ERR_ARG, "qw_codes / qw_scales is NULL");
  if ((uintptr_t)qw_codes % 16 != 0 || (format == RESQ_HIF4 && (uintptr_t)qw_scales % 4 != 0))
    return fail(RESQ_ERR_ARG, "qw_codes must be 16-byte aligned (HiF4 scales 4-byte aligned)");
  ActWs w{};
  const size_t act = carve_fwd(workspace, format, sp, m, d, n, &w);
  const size_t need = act + prepared_bytes(format, n, d);
  rc = check_ws(workspace, workspace_bytes, need);
  if (rc != RESQ_OK) return rc;
  hipStream_t s = (hipStream_t)stream;
  void* wprep = (char*)workspace + act;
  if (d > 0) {
    const uint8_t *frag, *fsc;
    carve_prepared(wprep, format, n, d, &frag, &fsc);
    resq::ProfScope prof_(resq::kProfPack, s);
    resq::launch_pack(b_pack_mode(format), qw_codes, qw_scales, n, d, (uint8_t*)frag, (uint8_t*)fsc, s);
  }
  return linear_fwd_core(format, sp, X, m, d, ldx, wprep, n, Y, ldy, false, w, s);
}

namespace {

int check_mixed_args(int format, const uint16_t* X, int64_t m, int64_t d, int64_t ldx, int64_t n,
                     const void* Y, int64_t ldy) {
  if (!valid_format(format)) return fail(RESQ_ERR_ARG, "unknown format %d", format);
  if (m < 0 || d < 0 || n < 0) return fail(RESQ_ERR_ARG, "negative size");
  if (ldx < d || ldy < n) return fail(RESQ_ERR_ARG, "ldx < d or ldy < n");
  if (d % block_of(format) != 0)
    return fail(RESQ_ERR_SHAPE, "d (%lld) is not a multiple of the block size %lld", (long long)d,
                (long long)block_of(format));
  if (m > 0 && n > 0 && !Y) return fail(RESQ_ERR_ARG, "Y is NULL");
  if (m > 0 && d > 0 && (!X || (uintptr_t)X % 16 != 0 || ldx % 8 != 0))
    return fail(RESQ_ERR_ARG, "X must be non-NULL, 16-byte aligned, with ldx %% 8 == 0");
  return ok();
}

}  // namespace

int resq_linear_w4a16(int format, const uint16_t* X, int64_t m, int64_t d, int64_t ldx,
                      const uint8_t* qw_codes, const void* qw_scales, int64_t n, float* Y,
                      int64_t ldy, void* stream) {
  int rc = check_mixed_args(format, X, m, d, ldx, n, Y, ldy);
  if (rc != RESQ_OK) return rc;
  if (m == 0 || n == 0) return ok();
  hipStream_t s = (hipStream_t)stream;
  if (d == 0) {
    if (ldy == n) resq::launch_zero_f32(Y, m * n, s);
    else return fail(RESQ_ERR_UNSUPPORTED, "d = 0 needs ldy == n");
    return check_launch("resq_linear_w4a16");
  }
  if (!qw_codes || !qw_scales || (uintptr_t)qw_codes % 16 != 0 ||
      (format == RESQ_HIF4 && (uintptr_t)qw_scales % 4 != 0))
    return fail(RESQ_ERR_ARG, "qw_codes must be 16-byte aligned (HiF4 scales 4-byte aligned)");
  if (!resq::mixed_gemm_supported(d, ldx, 0, true))
    return fail(RESQ_ERR_UNSUPPORTED, "d or ldx too large for 32-bit operand offsets");
  {
    resq::ProfScope prof_(resq::kProfMixed, s, true);
    resq::launch_mixed_gemm(format, m, n, d, X, ldx, qw_codes, qw_scales, nullptr, 0, Y, ldy, s);
  }
  return check_launch("resq_linear_w4a16");
}

int resq_linear_w16a4(int format, const uint16_t* X, int64_t m, int64_t d, int64_t ldx,
                      const uint16_t* W, int64_t ldw, int64_t n, float* Y, int64_t ldy,
                      void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_mixed_args(format, X, m, d, ldx, n, Y, ldy);
  if (rc != RESQ_OK) return rc;
  if (m == 0 || n == 0) return ok();
  hipStream_t s = (hipStream_t)stream;
  if (d == 0) {
    if (ldy == n) resq::launch_zero_f32(Y, m * n, s);
    else return fail(RESQ_ERR_UNSUPPORTED, "d = 0 needs ldy == n");
    return check_launch("resq_linear_w16a4");
  }
  if (!W || (uintptr_t)W % 16 != 0 || ldw % 8 != 0 || ldw < d)
    return fail(RESQ_ERR_ARG, "W must be non-NULL, 16-byte aligned, with ldw %% 8 == 0 and ldw >= d");
  if (!resq::mixed_gemm_supported(d, d, ldw, false))
    return fail(RESQ_ERR_UNSUPPORTED, "d or ldw too large for 32-bit operand offsets");
  rc = check_ws(workspace, workspace_bytes, align256((size_t)m * d * 2));
  if (rc != RESQ_OK) return rc;
  uint16_t* qx = (uint16_t*)workspace;  // Q(X) dequantized to bf16, m x d
  {
    resq::ProfScope prof_(resq::kProfQuantRows, s);
    resq::launch_quant_rows_bf16(format, X, m, d, ldx, qx, d, s);
  }
  {
    resq::ProfScope prof_(resq::kProfMixed, s, true);
    resq::launch_mixed_gemm(format, m, n, d, qx, d, nullptr, nullptr, W, ldw, Y, ldy, s);
  }
  return check_launch("resq_linear_w16a4");
}

int resq_diagnostics(int format, const uint16_t* X, int64_t m, int64_t d, int64_t ldx,
                     float outlier_threshold, double* stats, void* workspace,
                     size_t workspace_bytes, void* stream) {
  if (!valid_format(format)) return fail(RESQ_ERR_ARG, "unknown format %d", format);
  if (m < 0 || d < 0) return fail(RESQ_ERR_ARG, "negative size (m=%lld, d=%lld)", (long long)m, (long long)d);
  if (ldx < d) return fail(RESQ_ERR_ARG, "ldx (%lld) < d (%lld)", (long long)ldx, (long long)d);
  if (d % block_of(format) != 0)
    return fail(RESQ_ERR_SHAPE, "d (%lld) is not a multiple of the block size %lld", (long long)d, (long long)block_of(format));
  if (!stats) return fail(RESQ_ERR_ARG, "stats is NULL");
  if (m > 0 && d > 0 && !X) return fail(RESQ_ERR_ARG, "X is NULL");
  if ((uintptr_t)stats % 8 != 0) return fail(RESQ_ERR_ARG, "stats must be 8-byte aligned");
  int rc = check_ws(workspace, workspace_bytes, resq::diag_ws_bytes(m, d));
  if (rc != RESQ_OK) return rc;
  hipStream_t s = (hipStream_t)stream;
  {
    resq::ProfScope prof_(resq::kProfDiag, s, true);
    resq::launch_diagnostics(format, X, m, d, ldx, outlier_threshold, stats, (double*)workspace, s);
  }
  return check_launch("resq_diagnostics");
}

int resq_linear_bwd(int format, const uint16_t* dY, const uint16_t* X, const uint16_t* W,
                    int64_t m, int64_t d, int64_t n, float* dX, float* dW, void* workspace,
                    size_t workspace_bytes, void* stream) {
  if (!valid_format(format)) return fail(RESQ_ERR_ARG, "unknown format %d", format);
  if (m < 0 || d < 0 || n < 0) return fail(RESQ_ERR_ARG, "negative size");
  const int64_t B = block_of(format);
  if (dX && n % B != 0) return fail(RESQ_ERR_SHAPE, "dX needs n (%lld) %% %lld == 0", (long long)n, (long long)B);
  if (dW && m % B != 0) return fail(RESQ_ERR_SHAPE, "dW needs m (%lld) %% %lld == 0", (long long)m, (long long)B);
  if (d == 0) return ok();
  if (m == 0 || n == 0) {
    // an empty contraction: the gradient that still has elements is all zeros
    hipStream_t s = (hipStream_t)stream;
    if (m == 0 && dW) resq::launch_zero_f32(dW, n * d, s);
    if (n == 0 && dX) resq::launch_zero_f32(dX, m * d, s);
    return check_launch("resq_linear_bwd");
  }
  if (!dY || (dX && !W) || (dW && !X)) return fail(RESQ_ERR_ARG, "NULL input pointer");
  if ((dX && !resq::gemm_supported(format, m, d, n, 1)) ||
      (dW && !resq::gemm_supported(format, n, d, m, 1)))
    return fail(RESQ_ERR_UNSUPPORTED, "GEMM operands too large for 32-bit offsets");
  BwdWs w{};
  const size_t need = carve_bwd(workspace, format, m, d, n, &w);
  int rc = check_ws(workspace, workspace_bytes, need);
  if (rc != RESQ_OK) return rc;
  hipStream_t s = (hipStream_t)stream;
  // dW first when both are wanted: one pass over dY writes Q_m(dY)^T (for dW) and Q_n(dY)
  // (for dX, into its own buffer).
  const bool both = dX && dW;
  if (dW) {
    // dW[n][d] = Q_m(dY)^T [n][m] . (Q_m(X)^T [d][m])^T : contraction over m
    {
      resq::ProfScope prof_(resq::kProfQuantCols, s);
      resq::launch_quant_cols_frag(a_pack_mode(format), dY, m, n, n, w.fa, w.fa_sc, s,
                                   both ? w.fr : nullptr, both ? w.fr_sc : nullptr);
      resq::launch_quant_cols_frag(b_pack_mode(format), X, m, d, d, w.fb, w.fb_sc, s);
    }
    const uint8_t* af[2] = {w.fa, w.fa};
    const uint8_t* asc[2] = {w.fa_sc, w.fa_sc};
    const resq::GemmOperands op = gemm_operands(format, n, d, m, 1, af, asc, w.fb, w.fb_sc, dW, d);
    resq::ProfScope prof_(resq::kProfGemm, s, true);
    if (!resq::launch_gemm(op, s)) return fail(RESQ_ERR_UNSUPPORTED, "GEMM operand layout rejected");
  }
  if (dX) {
    // dX[m][d] = Q_n(dY)[m][n] . (Q_n(W)^T [d][n])^T : contraction over n
    if (!both) {
      resq::ProfScope prof_(resq::kProfQuantRows, s);
      resq::launch_residual(format, resq::kResidNone, dY, m, n, n, w.fr, w.fr_sc, nullptr, nullptr,
                            nullptr, nullptr, s, true);
    }
    {
      resq::ProfScope prof_(resq::kProfQuantCols, s);
      resq::launch_quant_cols_frag(b_pack_mode(format), W, n, d, d, w.fb, w.fb_sc, s);
    }
    const uint8_t* af[2] = {w.fr, w.fr};
    const uint8_t* asc[2] = {w.fr_sc, w.fr_sc};
    const resq::GemmOperands op = gemm_operands(format, m, d, n, 1, af, asc, w.fb, w.fb_sc, dX, d);
    resq::ProfScope prof_(resq::kProfGemm, s, true);
    if (!resq::launch_gemm(op, s)) return fail(RESQ_ERR_UNSUPPORTED, "GEMM operand layout rejected");
  }
  return check_launch("resq_linear_bwd");
}

}  // extern "C"
