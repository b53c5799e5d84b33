"""C ABI contract tests that need no GPU: the library loads, exports every entry point that
include/resq.h declares, and rejects bad arguments on the host before enqueueing anything."""
import ctypes
import os
import re

import pytest

import paper_2607_26515_amd as P
from paper_2607_26515_amd import resq as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "resq.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(resq_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(P.library_path())
    names = _declared()
    assert {"resq_quantize", "resq_residual_sparsify", "resq_linear_fwd", "resq_linear_bwd"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(B.EXPORTED)


def test_version_and_empty_error():
    assert P.resq_version().startswith("resq-gfx950")
    assert P.resq_workspace_size(B.OP_LINEAR_FWD, B.HIF4, B.S_2_4, 16, 2048, 2048) > 0


@pytest.mark.parametrize("args,code", [
    ((7, 0, 0, 4, 64, 64, 1, 0, 0), B.ERR_ARG),          # bad format
    ((0, 0, 3, 4, 64, 64, 1, 0, 0), B.ERR_ARG),          # bad dtype
    ((0, 0, 0, 4, 64, 64, 2, 0, 0), B.ERR_ARG),          # bad axis
    ((0, 0, 0, 4, 64, 32, 1, 0, 0), B.ERR_ARG),          # ld < cols
    ((0, 0, 0, 4, 48, 48, 1, 0, 0), B.ERR_SHAPE),        # 48 % 32 != 0 along the blocked axis
    ((1, 0, 0, 4, 96, 96, 1, 0, 0), B.ERR_SHAPE),        # 96 % 64 != 0 (HiF4)
    ((1, 0, 0, 96, 64, 64, 0, 0, 0), B.ERR_SHAPE),       # axis 0 blocks along rows
    ((0, 0, 0, 4, 64, 64, 1, 0, 0), B.ERR_ARG),          # NULL pointers
    ((0, 0, 0, -1, 64, 64, 1, 0, 0), B.ERR_ARG),         # negative size
])
def test_quantize_rejects_bad_arguments(args, code):
    assert P.resq_quantize(*args, 0) == code
    assert P.resq_last_error() != ""


def test_quantize_empty_is_ok():
    assert P.resq_quantize(0, 0, 0, 0, 64, 64, 1, 0, 0, 0) == B.OK
    assert P.resq_last_error() == ""


@pytest.mark.parametrize("fmt,sp,m,d,ldx,code", [
    (9, B.S_2_4, 4, 64, 64, B.ERR_ARG),
    (B.MXFP4, 11, 4, 64, 64, B.ERR_ARG),
    (B.MXFP4, B.S_2_4, 4, 64, 32, B.ERR_ARG),
    (B.HIF4, B.S_2_4, 4, 96, 96, B.ERR_SHAPE),
    (B.MXFP4, B.S_BLOCK32X64_50, 4, 96, 96, B.ERR_SHAPE),
    (B.MXFP4, B.S_2_4, 4, 64, 64, B.ERR_ARG),  # X NULL
])
def test_residual_sparsify_rejects_bad_arguments(fmt, sp, m, d, ldx, code):
    assert P.resq_residual_sparsify(fmt, sp, 0, m, d, ldx, 0, 0, 0, 0, 0, 0, 0, 0, 0) == code


@pytest.mark.parametrize("sp", [B.S_NM(0, 4), B.S_NM(4, 4), B.S_NM(2, 6), B.S_NM(8, 8),
                                B.S_CHANNEL(0), B.S_CHANNEL(100), B.S_BLOCK32X64(0),
                                B.S_UNSTRUCT(100), 0x500 | 50, 6, -1])
def test_invalid_sparsity_codes_are_rejected(sp):
    ptr = 1 << 20  # never dereferenced: the code is checked before anything else
    assert P.resq_residual_sparsify(B.MXFP4, sp, ptr, 4, 64, 64, ptr, ptr, ptr, ptr, 0, 0, 0, 0, 0) == B.ERR_ARG
    assert "sparsity" in P.resq_last_error()
    assert P.resq_workspace_size(B.OP_LINEAR_FWD_PREPARED, B.MXFP4, sp, 4, 64, 64) == 0


def test_parametric_codes_match_the_fifty_percent_kinds():
    """The parametric codes name the same functions: the 50% levels need the workspace of the
    50% kinds, other levels of a family the same, and the local patterns none for selection."""
    for op in (B.OP_RESIDUAL_SPARSIFY, B.OP_LINEAR_FWD_PREPARED):
        for kind, code in ((B.S_CHANNEL50, B.S_CHANNEL), (B.S_BLOCK32X64_50, B.S_BLOCK32X64),
                           (B.S_UNSTRUCT50, B.S_UNSTRUCT)):
            want = P.resq_workspace_size(op, B.HIF4, kind, 100, 2048, 256)
            assert want > 0
            for p in (1, 50, 99):
                assert P.resq_workspace_size(op, B.HIF4, code(p), 100, 2048, 256) == want
        want = P.resq_workspace_size(op, B.HIF4, B.S_2_4, 100, 2048, 256)
        for k, g in ((1, 4), (2, 4), (3, 4), (1, 8), (7, 8)):
            assert P.resq_workspace_size(op, B.HIF4, B.S_NM(k, g), 100, 2048, 256) == want
    assert B.sparsity_code("2:4") == B.S_2_4 and B.sparsity_code("3:8") == B.S_NM(3, 8)
    assert B.sparsity_code("channel25") == B.S_CHANNEL(25)
    assert B.sparsity_code("block32x64_75") == B.S_BLOCK32X64(75)
    assert B.sparsity_code("unstructured10") == B.S_UNSTRUCT(10)


def test_linear_fwd_rejects_bad_arguments():
    # ldy < n
    assert P.resq_linear_fwd(0, 2, 16, 4, 64, 64, 16, 16, 8, 16, 4, 0, 0, 0) == B.ERR_ARG
    # workspace missing (all pointers non-NULL and 256-aligned, but no workspace)
    assert P.resq_linear_fwd(0, 2, 256, 4, 64, 64, 256, 256, 8, 256, 8, 0, 0, 0) == B.ERR_WORKSPACE
    # misaligned workspace
    assert P.resq_linear_fwd(0, 2, 256, 4, 64, 64, 256, 256, 8, 256, 8, 257, 1 << 20, 0) == B.ERR_WORKSPACE
    # workspace too small
    assert P.resq_linear_fwd(0, 2, 256, 4, 64, 64, 256, 256, 8, 256, 8, 256, 16, 0) == B.ERR_WORKSPACE
    # Y NULL
    assert P.resq_linear_fwd(0, 2, 256, 4, 64, 64, 256, 256, 8, 0, 8, 256, 1 << 20, 0) == B.ERR_ARG


def test_linear_bwd_rejects_bad_arguments():
    # n not a multiple of the block for dX
    assert P.resq_linear_bwd(1, 256, 256, 256, 64, 64, 96, 256, 0, 256, 1 << 30, 0) == B.ERR_SHAPE
    # m not a multiple of the block for dW
    assert P.resq_linear_bwd(0, 256, 256, 256, 48, 64, 64, 0, 256, 256, 1 << 30, 0) == B.ERR_SHAPE
    assert P.resq_linear_bwd(0, 256, 256, 256, 64, 64, 64, 256, 256, 0, 0, 0) == B.ERR_WORKSPACE
    assert P.resq_linear_bwd(0, 0, 256, 256, 64, 64, 64, 256, 256, 256, 1 << 30, 0) == B.ERR_ARG


def test_workspace_sizes_grow_with_shape():
    a = P.resq_workspace_size(B.OP_LINEAR_FWD, B.HIF4, B.S_2_4, 256, 2048, 22016)
    b = P.resq_workspace_size(B.OP_LINEAR_FWD, B.HIF4, B.S_2_4, 512, 2048, 22016)
    assert 0 < a < b
    assert P.resq_workspace_size(9, 0, 0, 1, 64, 1) == 0
    assert P.resq_workspace_size(B.OP_LINEAR_BWD, B.MXFP4, 0, 64, 64, 64) > 0


def test_diagnostics_rejects_bad_arguments():
    ptr = 1 << 20  # never dereferenced
    assert P.resq_diagnostics(7, ptr, 4, 64, 64, 1.0, ptr, 0, 0, 0) == B.ERR_ARG
    assert P.resq_diagnostics(B.HIF4, ptr, 4, 96, 96, 1.0, ptr, 0, 0, 0) == B.ERR_SHAPE
    assert P.resq_diagnostics(B.MXFP4, ptr, 4, 64, 32, 1.0, ptr, 0, 0, 0) == B.ERR_ARG
    assert P.resq_diagnostics(B.MXFP4, ptr, 4, 64, 64, 1.0, 0, 0, 0, 0) == B.ERR_ARG
    assert P.resq_diagnostics(B.MXFP4, 0, 4, 64, 64, 1.0, ptr, 0, 0, 0) == B.ERR_ARG
    need = P.resq_workspace_size(B.OP_DIAGNOSTICS, B.MXFP4, 0, 4, 64, 0)
    assert need > 0
    assert P.resq_diagnostics(B.MXFP4, ptr, 4, 64, 64, 1.0, ptr, 0, 0, 0) == B.ERR_WORKSPACE
    assert P.resq_workspace_size(B.OP_DIAGNOSTICS, B.MXFP4, 0, 0, 64, 0) == 0


def test_swiglu_forward_rejects_bad_arguments():
    ptr = 1 << 20  # never dereferenced
    ws = P.resq_workspace_size(B.OP_LINEAR_FWD_PREPARED, B.MXFP4, B.S_2_4, 4, 64, 8)
    call = P.resq_linear_fwd_prepared_swiglu
    # bad input dtype, unknown sparsity, ld < d, NULL U, misaligned G, missing workspace
    assert call(B.MXFP4, B.S_2_4, ptr, ptr, 7, 4, 64, 64, 64, ptr, 8, ptr, 8, 0, 0, 0) == B.ERR_ARG
    assert call(B.MXFP4, 99, ptr, ptr, B.IN_BF16, 4, 64, 64, 64, ptr, 8, ptr, 8, 0, 0, 0) == B.ERR_ARG
    assert call(B.MXFP4, B.S_2_4, ptr, ptr, B.IN_BF16, 4, 64, 63, 64, ptr, 8, ptr, 8, 0, 0, 0) == B.ERR_ARG
    assert call(B.MXFP4, B.S_2_4, ptr, 0, B.IN_BF16, 4, 64, 64, 64, ptr, 8, ptr, 8, 0, 0, 0) == B.ERR_ARG
    assert call(B.MXFP4, B.S_2_4, ptr + 2, ptr, B.IN_F32, 4, 64, 64, 64, ptr, 8, ptr, 8, 0, 0, 0) == B.ERR_ARG
    assert call(B.HIF4, B.S_2_4, ptr, ptr, B.IN_BF16, 4, 96, 96, 96, ptr, 8, ptr, 8, 0, 0, 0) == B.ERR_SHAPE
    assert ws > 0
    assert call(B.MXFP4, B.S_2_4, ptr, ptr, B.IN_BF16, 4, 64, 64, 64, ptr, 8, ptr, 8, 0, 0, 0) == B.ERR_WORKSPACE
    # nothing to do: m = 0
    assert call(B.MXFP4, B.S_2_4, 0, 0, B.IN_BF16, 0, 64, 64, 64, 0, 8, 0, 8, 0, 0, 0) == B.OK


def test_rmsnorm_forward_rejects_bad_arguments():
    ptr = 1 << 20  # never dereferenced
    call = P.resq_linear_fwd_prepared_rmsnorm
    m, d, n = 4, 64, 8
    ws = P.resq_workspace_size(B.OP_LINEAR_FWD_RMSNORM, B.MXFP4, B.S_2_4, m, d, n)
    base = P.resq_workspace_size(B.OP_LINEAR_FWD_PREPARED, B.MXFP4, B.S_2_4, m, d, n)
    assert base + 4 * m <= ws < base + 4 * m + 512  # plus the per-row factors
    big = P.resq_workspace_size(B.OP_LINEAR_FWD_RMSNORM, B.HIF4, B.S_2_4, 5000, 2048, 2560)
    assert big >= P.resq_workspace_size(B.OP_LINEAR_FWD_PREPARED, B.HIF4, B.S_2_4, 5000, 2048, 2560) + 20000
    # eps: zero, below 2^-126, NaN, inf
    for eps in (0.0, 2.0**-127, float("nan"), float("inf"), -1e-6):
        assert call(B.MXFP4, B.S_2_4, ptr, m, d, d, ptr, eps, ptr, n, ptr, n, ptr, ws, 0) == B.ERR_ARG, eps
    # d beyond 2^18, NULL gamma, odd H address, ld < d, block size, missing workspace
    assert call(B.MXFP4, B.S_2_4, ptr, m, 2**18 + 32, 2**18 + 32, ptr, 1e-6, ptr, n, ptr, n, ptr, ws, 0) \
        == B.ERR_UNSUPPORTED
    assert call(B.MXFP4, B.S_2_4, ptr, m, d, d, 0, 1e-6, ptr, n, ptr, n, ptr, ws, 0) == B.ERR_ARG
    assert call(B.MXFP4, B.S_2_4, ptr + 1, m, d, d, ptr, 1e-6, ptr, n, ptr, n, ptr, ws, 0) == B.ERR_ARG
    assert call(B.MXFP4, B.S_2_4, ptr, m, d, d - 1, ptr, 1e-6, ptr, n, ptr, n, ptr, ws, 0) == B.ERR_ARG
    assert call(B.HIF4, B.S_2_4, ptr, m, 96, 96, ptr, 1e-6, ptr, n, ptr, n, ptr, ws, 0) == B.ERR_SHAPE
    assert call(B.MXFP4, B.S_2_4, ptr, m, d, d, ptr, 1e-6, ptr, n, ptr, n, 0, 0, 0) == B.ERR_WORKSPACE
    # nothing to do: m = 0
    assert call(B.MXFP4, B.S_2_4, 0, 0, d, d, 0, 1e-6, 0, n, 0, n, 0, 0, 0) == B.OK


def test_profiler_names_and_reset():
    import ctypes
    n, ms = ctypes.c_int64(-1), ctypes.c_double(-1.0)
    lib = P.load()
    P.resq_profile_enable(False)
    P.resq_profile_reset()
    for name in (b"residual", b"quant_rows", b"quant_cols", b"pack_hif4", b"select", b"gemm", b"diagnostics"):
        assert lib.resq_profile_read(name, ctypes.byref(n), ctypes.byref(ms)) == B.OK
        assert n.value == 0 and ms.value == 0.0
    assert lib.resq_profile_read(b"no_such_kernel", ctypes.byref(n), ctypes.byref(ms)) == B.ERR_ARG


def test_gemm_plan_query():
    info = (ctypes.c_int32 * 4)()
    assert P.resq_gemm_plan(B.MXFP4, 256, 2560, 2048, 1, info) == B.OK
    assert list(info) == [0, 1, 2, 4]
    assert P.resq_gemm_plan(5, 256, 2560, 2048, 1, info) == B.ERR_ARG
    assert P.resq_gemm_plan(B.MXFP4, -1, 2560, 2048, 1, info) == B.ERR_ARG
    assert P.gemm_plan("mxfp4", 8192, 37888, 3584) == {"tile": "128x256", "ksplit": 1, "kgroups": 1, "stages": 4}


def test_noalloc_rejects_oversized_calls_on_the_host():
    """resq_linear_fwd_prepared_noalloc checks its scratch need before any HIP call: sizes
    beyond RESQ_NOALLOC_SCRATCH_BYTES return RESQ_ERR_UNSUPPORTED (no GPU needed)."""
    ptr = 1 << 20  # never dereferenced
    m, d, n = 8192, 18944, 64
    need = P.resq_workspace_size(B.OP_LINEAR_FWD_PREPARED, B.HIF4, B.S_2_4, m, d, n)
    assert need > B.NOALLOC_SCRATCH_BYTES
    rc = P.resq_linear_fwd_prepared_noalloc(B.HIF4, B.S_2_4, ptr, m, d, d, ptr, n, ptr, n, 0)
    assert rc == B.ERR_UNSUPPORTED and "scratch" in P.resq_last_error()
    assert P.resq_linear_fwd_prepared_noalloc(B.HIF4, 99, ptr, 4, 64, 64, ptr, n, ptr, n, 0) == B.ERR_ARG
    assert P.resq_linear_fwd_prepared_noalloc(B.HIF4, B.S_2_4, ptr, 0, 64, 64, ptr, n, ptr, n, 0) == B.OK


def test_mixed_forms_check_arguments_on_the_host():
    ptr = 1 << 20  # 16-byte aligned, never dereferenced
    # misaligned X, ldx % 8 != 0, d not a multiple of the block, unknown format
    assert P.resq_linear_w4a16(B.MXFP4, ptr + 2, 4, 64, 64, ptr, ptr, 8, ptr, 8, 0) == B.ERR_ARG
    assert P.resq_linear_w4a16(B.MXFP4, ptr, 4, 64, 68, ptr, ptr, 8, ptr, 8, 0) == B.ERR_ARG
    assert P.resq_linear_w4a16(B.HIF4, ptr, 4, 96, 96, ptr, ptr, 8, ptr, 8, 0) == B.ERR_SHAPE
    assert P.resq_linear_w4a16(7, ptr, 4, 64, 64, ptr, ptr, 8, ptr, 8, 0) == B.ERR_ARG
    # W16A4: W row stride, missing workspace
    assert P.resq_linear_w16a4(B.MXFP4, ptr, 4, 64, 64, ptr, 60, 8, ptr, 8, ptr, 1 << 20, 0) == B.ERR_ARG
    assert P.resq_linear_w16a4(B.MXFP4, ptr, 4, 64, 64, ptr, 64, 8, ptr, 8, 0, 0, 0) == B.ERR_WORKSPACE
    # empty shapes are accepted without launching anything
    assert P.resq_linear_w4a16(B.HIF4, ptr, 0, 64, 64, ptr, ptr, 8, ptr, 8, 0) == B.OK
    # workspace: Q(X) as bf16 values, m x d (256-byte aligned)
    assert P.resq_workspace_size(B.OP_LINEAR_W16A4, B.HIF4, 0, 100, 128, 8) == 100 * 128 * 2
    assert P.resq_workspace_size(B.OP_LINEAR_W16A4, B.MXFP4, 0, 3, 96, 8) == 768
    # operand rows beyond the kernel's 32-bit offsets are refused before anything is enqueued
    assert P.resq_linear_w4a16(B.MXFP4, ptr, 4, 64, 1 << 31, ptr, ptr, 8, ptr, 8, 0) == B.ERR_UNSUPPORTED


def test_residual_sparsify_workspace_holds_block_partials():
    """The block kind's resq_residual_sparsify writes per-row scale-block sums (m x d / B
    doubles) into its workspace besides the keys; the size query counts them."""
    for fmt, blk in ((B.MXFP4, 32), (B.HIF4, 64)):
        for m, d in ((1, 64), (100, 2048), (512, 18944)):
            need = P.resq_workspace_size(B.OP_RESIDUAL_SPARSIFY, fmt, B.S_BLOCK32X64_50, m, d, 0)
            nblocks = -(-m // 32) * (d // 64)
            assert need >= m * (d // blk) * 8 + nblocks * 8, (fmt, m, d, need)
