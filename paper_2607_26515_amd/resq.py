"""Python binding of libresq.so (the C ABI declared in include/resq.h).

Two layers:

* ``resq_quantize``, ``resq_residual_sparsify``, ``resq_linear_fwd``, ``resq_linear_bwd``,
  ``resq_workspace_size``, ``resq_last_error``, ``resq_version``: the C entry points with the
  same names and arguments (integers for device pointers and the stream); they return the
  status code.
* ``quantize``, ``residual_sparsify``, ``linear_fwd``, ``linear_bwd``: the same calls on
  torch CUDA tensors.  They allocate outputs and the workspace with torch, pass pointers and
  the current stream, and raise ``ResqError`` on a non-zero status.  Every computation runs
  in the library's HIP kernels; nothing here touches the data.

The library must have been built (``python -m paper_2607_26515_amd.build``); importing a
function that needs it raises ``ResqError`` otherwise.  There is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libresq.so")
_lib = None

MXFP4, HIF4 = 0, 1
FORMATS = {"mxfp4": MXFP4, "hif4": HIF4}
S_NONE, S_IDENTITY, S_2_4, S_CHANNEL50, S_BLOCK32X64_50, S_UNSTRUCT50 = range(6)
SPARSITY = {"none": S_NONE, "identity": S_IDENTITY, "2:4": S_2_4, "channel50": S_CHANNEL50,
            "block32x64_50": S_BLOCK32X64_50, "unstructured50": S_UNSTRUCT50}


# Other levels and k:g patterns (the RESQ_S_NM / _CHANNEL / _BLOCK32X64 / _UNSTRUCT codes).
def S_NM(k, g):
    return 0x100 | (k << 4) | g


def S_CHANNEL(p):
    return 0x200 | p


def S_BLOCK32X64(p):
    return 0x300 | p


def S_UNSTRUCT(p):
    return 0x400 | p


def sparsity_code(name: str) -> int:
    """Library code of a sparsity name: the six names of SPARSITY, "k:g" (keep k of every g
    along d), "channel<p>", "block32x64_<p>" or "unstructured<p>" (keep p percent)."""
    if name in SPARSITY:
        return SPARSITY[name]
    if ":" in name:
        k, g = (int(v) for v in name.split(":"))
        return S_NM(k, g)
    for prefix, code in (("channel", S_CHANNEL), ("block32x64_", S_BLOCK32X64),
                         ("unstructured", S_UNSTRUCT)):
        if name.startswith(prefix) and name[len(prefix):].isdigit():
            return code(int(name[len(prefix):]))
    raise ValueError(f"unknown sparsity {name!r}")


def sparsity_family(code: int) -> str:
    """"none", "identity", "local", "channel", "block" or "unstructured" for a library code."""
    fam = {S_NONE: "none", S_IDENTITY: "identity", S_2_4: "local", S_CHANNEL50: "channel",
           S_BLOCK32X64_50: "block", S_UNSTRUCT50: "unstructured"}
    if code in fam:
        return fam[code]
    return {1: "local", 2: "channel", 3: "block", 4: "unstructured"}.get(code >> 8, "invalid")
OK, ERR_ARG, ERR_SHAPE, ERR_UNSUPPORTED, ERR_HIP, ERR_WORKSPACE = 0, -1, -2, -3, -4, -5
IN_BF16, IN_F32 = 0, 1
NOALLOC_SCRATCH_BYTES = 64 << 20  # RESQ_NOALLOC_SCRATCH_BYTES
OP_RESIDUAL_SPARSIFY, OP_LINEAR_FWD, OP_LINEAR_BWD, OP_LINEAR_FWD_PREPARED, OP_DIAGNOSTICS = 0, 1, 2, 3, 4
OP_LINEAR_W16A4 = 5
OP_LINEAR_FWD_RMSNORM = 6
DIAG_STATS = ("elements", "zeros_x", "zeros_qx", "blocks", "outlier_blocks", "energy_qx",
              "sse24_qx", "energy_qr", "sse24_qr")

EXPORTED = ("resq_quantize", "resq_residual_sparsify", "resq_linear_fwd", "resq_linear_bwd",
            "resq_workspace_size", "resq_last_error", "resq_version", "resq_profile_enable",
            "resq_profile_reset", "resq_profile_read", "resq_prepared_weights_size",
            "resq_prepare_weights", "resq_linear_fwd_prepared", "resq_linear_fwd_prepared_bf16",
            "resq_diagnostics", "resq_linear_fwd_prepared_swiglu", "resq_gemm_plan",
            "resq_linear_fwd_prepared_noalloc", "resq_linear_w4a16", "resq_linear_w16a4",
            "resq_linear_fwd_prepared_rmsnorm")
GEMM_TILES = {0: "64x64", 1: "128x256", 2: "128x192", 3: "128x192_8w", 4: "64x128"}


class ResqError(RuntimeError):
    def __init__(self, msg: str, code: int = 0):
        super().__init__(msg)
        self.code = code


def library_path() -> str:
    return _LIB_PATH


def load() -> ctypes.CDLL:
    """Load libresq.so once (raises ResqError if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ResqError(f"{_LIB_PATH} is missing: build it with `python -m paper_2607_26515_amd.build`")
    # PyTorch ships its own HIP runtime.  Loaded first, it is the one the library binds to
    # (same soname); loaded after the library, it comes in as a second copy beside the
    # system one, and the library's launches then find no device.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
    lib.resq_quantize.argtypes = [i32, vp, i32, i64, i64, i64, i32, vp, vp, vp]
    lib.resq_residual_sparsify.argtypes = [i32, i32, vp, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.resq_linear_fwd.argtypes = [i32, i32, vp, i64, i64, i64, vp, vp, i64, vp, i64, vp, sz, vp]
    lib.resq_linear_bwd.argtypes = [i32, vp, vp, vp, i64, i64, i64, vp, vp, vp, sz, vp]
    lib.resq_workspace_size.argtypes = [i32, i32, i32, i64, i64, i64]
    lib.resq_prepared_weights_size.argtypes = [i32, i64, i64]
    lib.resq_prepared_weights_size.restype = sz
    lib.resq_prepare_weights.argtypes = [i32, vp, vp, i64, i64, vp, vp]
    lib.resq_prepare_weights.restype = i32
    lib.resq_linear_fwd_prepared.argtypes = [i32, i32, vp, i64, i64, i64, vp, i64, vp, i64, vp, sz, vp]
    lib.resq_linear_fwd_prepared.restype = i32
    lib.resq_linear_fwd_prepared_bf16.argtypes = [i32, i32, vp, i64, i64, i64, vp, i64, vp, i64, vp, sz, vp]
    lib.resq_linear_fwd_prepared_bf16.restype = i32
    lib.resq_diagnostics.argtypes = [i32, vp, i64, i64, i64, ctypes.c_float, vp, vp, sz, vp]
    lib.resq_diagnostics.restype = i32
    lib.resq_linear_fwd_prepared_swiglu.argtypes = [i32, i32, vp, vp, i32, i64, i64, i64, i64, vp, i64,
                                                    vp, i64, vp, sz, vp]
    lib.resq_linear_fwd_prepared_swiglu.restype = i32
    lib.resq_linear_fwd_prepared_rmsnorm.argtypes = [i32, i32, vp, i64, i64, i64, vp, ctypes.c_float,
                                                     vp, i64, vp, i64, vp, sz, vp]
    lib.resq_linear_fwd_prepared_rmsnorm.restype = i32
    for f in ("resq_quantize", "resq_residual_sparsify", "resq_linear_fwd", "resq_linear_bwd"):
        getattr(lib, f).restype = i32
    lib.resq_workspace_size.restype = sz
    lib.resq_profile_enable.argtypes = [i32]
    lib.resq_profile_enable.restype = i32
    lib.resq_profile_reset.argtypes = []
    lib.resq_profile_reset.restype = None
    lib.resq_profile_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(i64), ctypes.POINTER(ctypes.c_double)]
    lib.resq_profile_read.restype = i32
    lib.resq_linear_fwd_prepared_noalloc.argtypes = [i32, i32, vp, i64, i64, i64, vp, i64, vp, i64, vp]
    lib.resq_linear_fwd_prepared_noalloc.restype = i32
    lib.resq_linear_w4a16.argtypes = [i32, vp, i64, i64, i64, vp, vp, i64, vp, i64, vp]
    lib.resq_linear_w4a16.restype = i32
    lib.resq_linear_w16a4.argtypes = [i32, vp, i64, i64, i64, vp, i64, i64, vp, i64, vp, sz, vp]
    lib.resq_linear_w16a4.restype = i32
    lib.resq_gemm_plan.argtypes = [i32, i64, i64, i64, i32, ctypes.POINTER(ctypes.c_int32)]
    lib.resq_gemm_plan.restype = i32
    lib.resq_last_error.restype = ctypes.c_char_p
    lib.resq_version.restype = ctypes.c_char_p
    _lib = lib
    return lib


# ------------------------------------------------------------------------------------------
# C entry points (pointers and the stream as integers; 0 = NULL / default stream)
# ------------------------------------------------------------------------------------------
def resq_quantize(fmt, x, in_dtype, rows, cols, ld, axis, codes, scales, stream=0) -> int:
    return load().resq_quantize(fmt, x, in_dtype, rows, cols, ld, axis, codes, scales, stream)


def resq_residual_sparsify(fmt, sparsity, X, m, d, ldx, qx_codes, qx_scales, qr_codes, qr_scales,
                           keep_mask, group_mask, workspace, workspace_bytes, stream=0) -> int:
    return load().resq_residual_sparsify(fmt, sparsity, X, m, d, ldx, qx_codes, qx_scales, qr_codes,
                                         qr_scales, keep_mask, group_mask, workspace,
                                         workspace_bytes, stream)


def resq_linear_fwd(fmt, sparsity, X, m, d, ldx, qw_codes, qw_scales, n, Y, ldy, workspace,
                    workspace_bytes, stream=0) -> int:
    return load().resq_linear_fwd(fmt, sparsity, X, m, d, ldx, qw_codes, qw_scales, n, Y, ldy,
                                  workspace, workspace_bytes, stream)


def resq_linear_bwd(fmt, dY, X, W, m, d, n, dX, dW, workspace, workspace_bytes, stream=0) -> int:
    return load().resq_linear_bwd(fmt, dY, X, W, m, d, n, dX, dW, workspace, workspace_bytes, stream)


def resq_prepared_weights_size(fmt, n, d) -> int:
    return load().resq_prepared_weights_size(fmt, n, d)


def resq_prepare_weights(fmt, qw_codes, qw_scales, n, d, wprep, stream=0) -> int:
    return load().resq_prepare_weights(fmt, qw_codes, qw_scales, n, d, wprep, stream)


def resq_linear_fwd_prepared(fmt, sparsity, X, m, d, ldx, wprep, n, Y, ldy, workspace,
                             workspace_bytes, stream=0) -> int:
    return load().resq_linear_fwd_prepared(fmt, sparsity, X, m, d, ldx, wprep, n, Y, ldy,
                                           workspace, workspace_bytes, stream)


def resq_linear_fwd_prepared_noalloc(fmt, sparsity, X, m, d, ldx, wprep, n, Y, ldy, stream=0) -> int:
    return load().resq_linear_fwd_prepared_noalloc(fmt, sparsity, X, m, d, ldx, wprep, n, Y, ldy, stream)


def resq_linear_w4a16(fmt, X, m, d, ldx, qw_codes, qw_scales, n, Y, ldy, stream=0) -> int:
    return load().resq_linear_w4a16(fmt, X, m, d, ldx, qw_codes, qw_scales, n, Y, ldy, stream)


def resq_linear_w16a4(fmt, X, m, d, ldx, W, ldw, n, Y, ldy, workspace, workspace_bytes, stream=0) -> int:
    return load().resq_linear_w16a4(fmt, X, m, d, ldx, W, ldw, n, Y, ldy, workspace, workspace_bytes,
                                    stream)


def resq_linear_fwd_prepared_bf16(fmt, sparsity, X, m, d, ldx, wprep, n, Y, ldy, workspace,
                                  workspace_bytes, stream=0) -> int:
    return load().resq_linear_fwd_prepared_bf16(fmt, sparsity, X, m, d, ldx, wprep, n, Y, ldy,
                                                workspace, workspace_bytes, stream)


def resq_linear_fwd_prepared_swiglu(fmt, sparsity, G, U, in_dtype, m, d, ldg, ldu, wprep, n, Y, ldy,
                                    workspace, workspace_bytes, stream=0) -> int:
    return load().resq_linear_fwd_prepared_swiglu(fmt, sparsity, G, U, in_dtype, m, d, ldg, ldu,
                                                  wprep, n, Y, ldy, workspace, workspace_bytes, stream)


def resq_linear_fwd_prepared_rmsnorm(fmt, sparsity, H, m, d, ldh, gamma, eps, wprep, n, Y, ldy,
                                     workspace, workspace_bytes, stream=0) -> int:
    return load().resq_linear_fwd_prepared_rmsnorm(fmt, sparsity, H, m, d, ldh, gamma, eps, wprep,
                                                   n, Y, ldy, workspace, workspace_bytes, stream)


def resq_diagnostics(fmt, X, m, d, ldx, outlier_threshold, stats, workspace, workspace_bytes,
                     stream=0) -> int:
    return load().resq_diagnostics(fmt, X, m, d, ldx, outlier_threshold, stats, workspace,
                                   workspace_bytes, stream)


def resq_gemm_plan(fmt, M, N, K, split_allowed, info) -> int:
    return load().resq_gemm_plan(fmt, M, N, K, split_allowed, info)


def gemm_plan(fmt, M, N, K, split_allowed=True):
    """The GEMM plan for Y[M][N] over K: dict(tile, ksplit, kgroups, stages) (host query)."""
    info = (ctypes.c_int32 * 4)()
    _check(resq_gemm_plan(_fmt(fmt), M, N, K, 1 if split_allowed else 0, info), "resq_gemm_plan")
    return {"tile": GEMM_TILES[info[0]], "ksplit": info[1], "kgroups": info[2], "stages": info[3]}


def resq_workspace_size(op, fmt, sparsity, m, d, n) -> int:
    return load().resq_workspace_size(op, fmt, sparsity, m, d, n)


def resq_last_error() -> str:
    return load().resq_last_error().decode()


def resq_version() -> str:
    return load().resq_version().decode()


def resq_profile_enable(on: bool) -> int:
    return load().resq_profile_enable(1 if on else 0)


def resq_profile_reset() -> None:
    load().resq_profile_reset()


def resq_profile_read(name: str):
    """(launches, total milliseconds) of a kernel family since the last reset."""
    n = ctypes.c_int64(0)
    ms = ctypes.c_double(0.0)
    rc = load().resq_profile_read(name.encode(), ctypes.byref(n), ctypes.byref(ms))
    _check(rc, "resq_profile_read")
    return n.value, ms.value


# ------------------------------------------------------------------------------------------
# torch helpers (argument marshalling only)
# ------------------------------------------------------------------------------------------
def _fmt(fmt) -> int:
    return FORMATS[fmt] if isinstance(fmt, str) else int(fmt)


def _sp(sp) -> int:
    return sparsity_code(sp) if isinstance(sp, str) else int(sp)


def _p(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream(stream) -> int:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream)


def _check(rc: int, what: str):
    if rc != OK:
        raise ResqError(f"{what} failed ({rc}): {resq_last_error()}", rc)


def _empty_u8(n, device):
    import torch
    return torch.empty(int(n), dtype=torch.uint8, device=device)


def scale_shape(fmt, outer, K):
    """(shape, dtype name) of the scale array of a K-major quantized tensor."""
    return ((outer, K // 32), "uint8") if _fmt(fmt) == MXFP4 else ((outer, K // 64), "int32")


def _empty_scales(fmt, outer, K, device):
    import torch
    shape, dt = scale_shape(fmt, outer, K)
    return torch.empty(shape, dtype=torch.uint8 if dt == "uint8" else torch.int32, device=device)


def workspace(op, fmt, sparsity, m, d, n=0, device="cuda"):
    import torch
    nb = resq_workspace_size(op, _fmt(fmt), _sp(sparsity), m, d, n)
    # torch's caching allocator returns 256-byte aligned blocks
    return torch.empty(max(nb, 1), dtype=torch.uint8, device=device), nb


def quantize(x, fmt, axis: int = 1, stream=None):
    """Q(x) in blocks along `axis` (1: along columns; 0: along rows, output transposed)."""
    import torch
    rows, cols = x.shape
    f32 = x.dtype == torch.float32
    if not f32 and x.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
        raise TypeError("x must be bfloat16 (or its uint16 bits) or float32")
    outer, K = (rows, cols) if axis == 1 else (cols, rows)
    codes = torch.empty((outer, K // 2), dtype=torch.uint8, device=x.device)
    scales = _empty_scales(fmt, outer, K, x.device)
    rc = resq_quantize(_fmt(fmt), _p(x), IN_F32 if f32 else IN_BF16, rows, cols, x.stride(0), axis,
                       _p(codes), _p(scales), _stream(stream))
    _check(rc, "resq_quantize")
    return codes, scales


def residual_sparsify(x, fmt, sparsity, stream=None):
    """Q(X), S(Q(X - Q(X))) and the masks, as a dict of device tensors."""
    import torch
    m, d = x.shape
    f, sp = _fmt(fmt), _sp(sparsity)
    out = {
        "qx_codes": torch.empty((m, d // 2), dtype=torch.uint8, device=x.device),
        "qx_scales": _empty_scales(f, m, d, x.device),
    }
    fam = sparsity_family(sp)
    if sp != S_NONE:
        out["qr_codes"] = torch.empty((m, d // 2), dtype=torch.uint8, device=x.device)
        out["qr_scales"] = _empty_scales(f, m, d, x.device)
        out["keep_mask"] = torch.empty((m, d // 8), dtype=torch.uint8, device=x.device)
    if fam == "channel":
        out["group_mask"] = torch.zeros(((d + 7) // 8,), dtype=torch.uint8, device=x.device)
    elif fam == "block":
        nblk = ((m + 31) // 32) * (d // 64)
        out["group_mask"] = torch.zeros(((nblk + 7) // 8,), dtype=torch.uint8, device=x.device)
    ws, nb = workspace(OP_RESIDUAL_SPARSIFY, f, sp, m, d, 0, x.device)
    rc = resq_residual_sparsify(f, sp, _p(x), m, d, x.stride(0), _p(out["qx_codes"]),
                                _p(out["qx_scales"]), _p(out.get("qr_codes")),
                                _p(out.get("qr_scales")), _p(out.get("keep_mask")),
                                _p(out.get("group_mask")), _p(ws), nb, _stream(stream))
    _check(rc, "resq_residual_sparsify")
    return out


def linear_fwd(x, qw_codes, qw_scales, fmt, sparsity, y=None, ws=None, stream=None):
    """Y = Q(X) Q(W)^T + S(Q(X - Q(X))) Q(W)^T (float32)."""
    import torch
    m, d = x.shape
    n = qw_codes.shape[0]
    f, sp = _fmt(fmt), _sp(sparsity)
    if y is None:
        y = torch.empty((m, n), dtype=torch.float32, device=x.device)
    if ws is None:
        ws = workspace(OP_LINEAR_FWD, f, sp, m, d, n, x.device)
    buf, nb = ws
    rc = resq_linear_fwd(f, sp, _p(x), m, d, x.stride(0), _p(qw_codes), _p(qw_scales), n, _p(y),
                         y.stride(0), _p(buf), nb, _stream(stream))
    _check(rc, "resq_linear_fwd")
    return y


def prepare_weights(qw_codes, qw_scales, fmt, stream=None):
    """Q(W) (K-major codes + scales) -> the GEMM's prepared weight operand (device tensor)."""
    import torch
    n, d = qw_codes.shape[0], qw_codes.shape[1] * 2
    f = _fmt(fmt)
    nb = resq_prepared_weights_size(f, n, d)
    wprep = torch.empty(max(nb, 1), dtype=torch.uint8, device=qw_codes.device)
    rc = resq_prepare_weights(f, _p(qw_codes), _p(qw_scales), n, d, _p(wprep), _stream(stream))
    _check(rc, "resq_prepare_weights")
    return wprep


def linear_fwd_prepared(x, wprep, n, fmt, sparsity, y=None, ws=None, stream=None, out="f32"):
    """Y = Q(X) Q(W)^T + S(Q(X - Q(X))) Q(W)^T with Q(W) in prepared form: float32, or with
    out="bf16" the bf16 rounding of the float32 result (returned as an int16 tensor of bf16
    bit patterns)."""
    import torch
    m, d = x.shape
    f, sp = _fmt(fmt), _sp(sparsity)
    if out not in ("f32", "bf16"):
        raise ValueError(f"out must be 'f32' or 'bf16', not {out!r}")
    if y is None:
        y = torch.empty((m, n), dtype=torch.float32 if out == "f32" else torch.int16, device=x.device)
    if ws is None:
        ws = workspace(OP_LINEAR_FWD_PREPARED, f, sp, m, d, n, x.device)
    buf, nb = ws
    call = resq_linear_fwd_prepared if out == "f32" else resq_linear_fwd_prepared_bf16
    rc = call(f, sp, _p(x), m, d, x.stride(0), _p(wprep), n, _p(y), y.stride(0), _p(buf), nb,
              _stream(stream))
    _check(rc, call.__name__)
    return y


def linear_bwd(dy, x, w, fmt, want_dx=True, want_dw=True, ws=None, stream=None):
    """dX = Q_n(dY) Q_n(W), dW = Q_m(dY)^T Q_m(X) (float32)."""
    import torch
    m, n = dy.shape
    d = x.shape[1]
    f = _fmt(fmt)
    dx = torch.empty((m, d), dtype=torch.float32, device=dy.device) if want_dx else None
    dw = torch.empty((n, d), dtype=torch.float32, device=dy.device) if want_dw else None
    if ws is None:
        ws = workspace(OP_LINEAR_BWD, f, S_NONE, m, d, n, dy.device)
    buf, nb = ws
    rc = resq_linear_bwd(f, _p(dy), _p(x), _p(w), m, d, n, _p(dx), _p(dw), _p(buf), nb,
                         _stream(stream))
    _check(rc, "resq_linear_bwd")
    return dx, dw


def linear_w4a16(x, qw_codes, qw_scales, fmt, y=None, stream=None):
    """Weight-only FP4 (Table 1, W4A16): Y = X Q(W)^T, X bf16, Q(W) K-major (float32 Y)."""
    import torch
    m, d = x.shape
    n = qw_codes.shape[0]
    if y is None:
        y = torch.empty((m, n), dtype=torch.float32, device=x.device)
    rc = resq_linear_w4a16(_fmt(fmt), _p(x), m, d, x.stride(0), _p(qw_codes), _p(qw_scales), n,
                           _p(y), y.stride(0), _stream(stream))
    _check(rc, "resq_linear_w4a16")
    return y


def linear_w16a4(x, w, fmt, y=None, ws=None, stream=None):
    """Activation-only FP4 (Table 1, W16A4): Y = Q(X) W^T, W bf16 (float32 Y)."""
    import torch
    m, d = x.shape
    n = w.shape[0]
    f = _fmt(fmt)
    if y is None:
        y = torch.empty((m, n), dtype=torch.float32, device=x.device)
    if ws is None:
        ws = workspace(OP_LINEAR_W16A4, f, S_NONE, m, d, n, x.device)
    buf, nb = ws
    rc = resq_linear_w16a4(f, _p(x), m, d, x.stride(0), _p(w), w.stride(0), n, _p(y), y.stride(0),
                           _p(buf), nb, _stream(stream))
    _check(rc, "resq_linear_w16a4")
    return y


def linear_fwd_rmsnorm(h, gamma, eps, wprep, n, fmt, sparsity, y=None, ws=None, stream=None):
    """Y = ResQ linear of X = RMSNorm(H) * gamma (formed inside the quantization pass); H is an
    m x d bf16 view (int16 bit patterns or bfloat16) with unit column stride, gamma d bf16
    values, eps a float32 >= 2^-126."""
    import torch
    m, d = h.shape
    f, sp = _fmt(fmt), _sp(sparsity)
    if gamma.numel() != d or not gamma.is_contiguous():
        raise ValueError("gamma must hold d contiguous values")
    if y is None:
        y = torch.empty((m, n), dtype=torch.float32, device=h.device)
    if ws is None:
        ws = workspace(OP_LINEAR_FWD_RMSNORM, f, sp, m, d, n, h.device)
    buf, nb = ws
    rc = resq_linear_fwd_prepared_rmsnorm(f, sp, _p(h), m, d, h.stride(0), _p(gamma), float(eps),
                                          _p(wprep), n, _p(y), y.stride(0), _p(buf), nb,
                                          _stream(stream))
    _check(rc, "resq_linear_fwd_prepared_rmsnorm")
    return y


def diagnostics(x, fmt, outlier_threshold, stream=None):
    """The Figs. 2-4 statistics of activations x (m x d bf16) as a float64 device tensor of
    len(DIAG_STATS) values, in the order of DIAG_STATS."""
    import torch
    m, d = x.shape
    f = _fmt(fmt)
    stats = torch.empty(len(DIAG_STATS), dtype=torch.float64, device=x.device)
    ws, nb = workspace(OP_DIAGNOSTICS, f, S_NONE, m, d, 0, x.device)
    rc = resq_diagnostics(f, _p(x), m, d, x.stride(0), float(outlier_threshold), _p(stats), _p(ws),
                          nb, _stream(stream))
    _check(rc, "resq_diagnostics")
    return stats


def linear_fwd_swiglu(g, u, wprep, n, fmt, sparsity, y=None, ws=None, stream=None):
    """Y = ResQ linear of X = silu(G) * U (bf16-rounded, formed inside the quantization pass);
    G and U are m x d bf16 (int16 bit patterns or bfloat16) or float32 views with unit column
    stride and the same dtype."""
    import torch
    m, d = g.shape
    f, sp = _fmt(fmt), _sp(sparsity)
    if g.dtype != u.dtype or g.shape != u.shape:
        raise ValueError("G and U must have the same shape and dtype")
    in_dtype = IN_F32 if g.dtype == torch.float32 else IN_BF16
    if y is None:
        y = torch.empty((m, n), dtype=torch.float32, device=g.device)
    if ws is None:
        ws = workspace(OP_LINEAR_FWD_PREPARED, f, sp, m, d, n, g.device)
    buf, nb = ws
    rc = resq_linear_fwd_prepared_swiglu(f, sp, _p(g), _p(u), in_dtype, m, d, g.stride(0), u.stride(0),
                                         _p(wprep), n, _p(y), y.stride(0), _p(buf), nb, _stream(stream))
    _check(rc, "resq_linear_fwd_prepared_swiglu")
    return y
