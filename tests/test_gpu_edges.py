"""Degenerate shapes on the GPU: empty row or column counts, and empty contractions (d = 0
in the forward, m = 0 or n = 0 in the backward), whose outputs are sums over nothing, i.e.
zeros."""
import numpy as np
import pytest

from synth import activations, grad_output, rng_tree, weights
from _gpu_util import dev_bf16, host, log

pytestmark = pytest.mark.gpu

FMTS = ["mxfp4", "hif4"]


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["none", "2:4", "identity", "channel50", "unstructured50"])
def test_forward_empty_contraction_gives_zeros(fmt, sp):
    import torch
    import paper_2607_26515_amd as P
    log(f"forward d=0 {fmt} {sp}")
    m, n = 37, 70
    x = torch.zeros((m, 0), dtype=torch.int16, device="cuda")
    w = torch.zeros((n, 0), dtype=torch.int16, device="cuda")
    qc, qs = P.quantize(w, fmt, axis=1)
    y1 = P.linear_fwd(x, qc, qs, fmt, sp, y=torch.full((m, n), 7.0, dtype=torch.float32, device="cuda"))
    y2 = P.linear_fwd_prepared(x, P.prepare_weights(qc, qs, fmt), n, fmt, sp,
                               y=torch.full((m, n), 7.0, dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    assert not host(y1).any() and not host(y2).any()


@pytest.mark.parametrize("fmt", FMTS)
def test_forward_empty_rows_or_columns(fmt):
    import torch
    import paper_2607_26515_amd as P
    log(f"forward m=0 / n=0 {fmt}")
    d = 128
    wb = weights(rng_tree(1, 1)[0], 64, d)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    wp = P.prepare_weights(qc, qs, fmt)
    y = P.linear_fwd_prepared(torch.zeros((0, d), dtype=torch.int16, device="cuda"), wp, 64, fmt, "2:4")
    assert y.shape == (0, 64)
    xb = activations(rng_tree(2, 1)[0], 5, d, 0.01, 50.0)
    y = P.linear_fwd_prepared(dev_bf16(xb), wp, 0, fmt, "2:4")
    torch.cuda.synchronize()
    assert y.shape == (5, 0)


@pytest.mark.parametrize("fmt", FMTS)
def test_backward_empty_contractions_give_zeros(fmt):
    """m = 0: dW = Q(dY)^T Q(X) sums over no rows; n = 0: dX = Q(dY) Q(W) sums over no
    output features.  Both are written as zeros over outputs that held other values."""
    import torch
    import paper_2607_26515_amd as P
    log(f"backward empty contractions {fmt}")
    d, n, m = 96, 64, 64
    lib = P.load()
    f = P.FORMATS[fmt]
    # m = 0: dW (n x d) must be zeroed
    w = dev_bf16(weights(rng_tree(3, 1)[0], n, d))
    dw = torch.full((n, d), 3.0, dtype=torch.float32, device="cuda")
    rc = lib.resq_linear_bwd(f, int(w.data_ptr()), int(w.data_ptr()), int(w.data_ptr()), 0, d, n, 0,
                             int(dw.data_ptr()), 0, 0, 0)
    torch.cuda.synchronize()
    assert rc == 0 and not host(dw).any()
    # n = 0: dX (m x d) must be zeroed
    x = dev_bf16(activations(rng_tree(4, 1)[0], m, d, 0.01, 50.0))
    dx = torch.full((m, d), 3.0, dtype=torch.float32, device="cuda")
    rc = lib.resq_linear_bwd(f, int(x.data_ptr()), int(x.data_ptr()), int(x.data_ptr()), m, d, 0,
                             int(dx.data_ptr()), 0, 0, 0, 0)
    torch.cuda.synchronize()
    assert rc == 0 and not host(dx).any()
    # the regular path right after, on the same stream, still matches a direct call
    gb = grad_output(rng_tree(5, 1)[0], m, n)
    a, b = P.linear_bwd(dev_bf16(gb), x, w, fmt)
    c, e = P.linear_bwd(dev_bf16(gb), x, w, fmt)
    torch.cuda.synchronize()
    assert torch.equal(a, c) and torch.equal(b, e)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("m,d,n", [(256, 2048, 2560), (256, 11008, 2048)])  # the second splits K
def test_profiler_counts_launch_families(fmt, m, d, n):
    """The library profiler sees one residual pass and one GEMM family interval per forward
    call (a K split's reduction is inside the GEMM's interval), with positive durations."""
    import torch
    import paper_2607_26515_amd as P
    log(f"profiler {fmt} m={m} d={d} n={n}")
    xb, wb = activations(rng_tree(6, 1)[0], m, d, 0.01, 50.0), weights(rng_tree(7, 1)[0], n, d)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    wp = P.prepare_weights(qc, qs, fmt)
    x = dev_bf16(xb)
    P.linear_fwd_prepared(x, wp, n, fmt, "2:4")
    torch.cuda.synchronize()
    P.resq_profile_enable(True)
    P.resq_profile_reset()
    for _ in range(3):
        P.linear_fwd_prepared(x, wp, n, fmt, "2:4")
    torch.cuda.synchronize()
    g, r = P.resq_profile_read("gemm"), P.resq_profile_read("residual")
    P.resq_profile_enable(False)
    assert g[0] == 3 and r[0] == 3
    assert 0.0 < g[1] < 3 * 10.0 and 0.0 < r[1] < 3 * 10.0  # milliseconds


def test_library_loaded_before_torch_still_launches():
    """A process that queries the library on the host before it imports PyTorch (here the
    plan query) must still launch kernels afterwards: the binding loads PyTorch's HIP runtime
    before the library, so the process holds one HIP runtime, not two.  Run in a fresh
    process, since this one has long loaded both."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = (
        "import paper_2607_26515_amd as P\n"
        "P.gemm_plan('mxfp4', 256, 2560, 2048)\n"
        "import torch\n"
        "w = torch.zeros((64, 64), dtype=torch.int16, device='cuda')\n"
        "c, s = P.quantize(w, 'mxfp4', axis=1)\n"
        "torch.cuda.synchronize()\n"
        "print('ok', int(c.sum()))\n"
    )
    log("library before torch, fresh process")
    r = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "ok 0" in r.stdout, r.stdout + r.stderr
