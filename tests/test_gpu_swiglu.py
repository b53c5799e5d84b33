"""GPU parity of the forward with the SwiGLU producer fused into the quantization pass
(resq_linear_fwd_prepared_swiglu): X = silu(G) * U is formed on the fly and rounded once to
bf16.  With X computed by the oracle and passed to the plain prepared forward, Y must be the
same bit for bit (same Q(X), dX, S and GEMM), and it must match the oracle's Y."""
import numpy as np
import pytest

from oracle import resq as Q
from synth import activations, bf16_bits_to_f32, f32_to_bf16_bits, rng_tree, weights
from _gpu_util import assert_close, dev_bf16, dev_f32, host, log

pytestmark = pytest.mark.gpu

FMTS = ["mxfp4", "hif4"]


def _inputs(m, d, seed, f32):
    rg, ru = rng_tree(seed, 2)
    g = bf16_bits_to_f32(activations(rg, m, d, 0.01, 8.0)) * np.float32(2.0)
    u = bf16_bits_to_f32(activations(ru, m, d, 0.01, 30.0))
    if f32:  # values off the bf16 grid
        g = g * np.float32(1.0 + 2.0**-12)
        u = u * np.float32(1.0 - 2.0**-11)
    else:
        g, u = bf16_bits_to_f32(f32_to_bf16_bits(g)), bf16_bits_to_f32(f32_to_bf16_bits(u))
    return g.astype(np.float32), u.astype(np.float32)


def _dev(a, f32):
    return dev_f32(a) if f32 else dev_bf16(f32_to_bf16_bits(a))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["none", "2:4", "4:8", "channel50", "unstructured50"])
@pytest.mark.parametrize("f32", [False, True])
@pytest.mark.parametrize("m,d,n,layout", [(37, 512, 100, "concat"), (100, 2048, 300, "separate"),
                                          (256, 11008, 512, "concat"), (33, 640, 64, "strided")])
def test_swiglu_forward(fmt, sp, f32, m, d, n, layout):
    import torch
    import paper_2607_26515_amd as P
    log(f"swiglu {fmt} {sp} f32={f32} m={m} d={d} n={n} {layout}")
    g, u = _inputs(m, d, seed=m + d + n, f32=f32)
    if layout == "concat":  # one [gate | up] buffer, row stride 2d
        base = _dev(np.concatenate([g, u], axis=1), f32)
        gd, ud = base[:, :d], base[:, d:]
    elif layout == "strided":  # row stride d + 1: the scalar load path
        gd = _dev(np.pad(g, ((0, 0), (0, 1))), f32)[:, :d]
        ud = _dev(np.pad(u, ((0, 0), (0, 1))), f32)[:, :d]
    else:
        gd, ud = _dev(g, f32), _dev(u, f32)
    wb = weights(rng_tree(n, 1)[0], n, d)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    wprep = P.prepare_weights(qc, qs, fmt)
    y = host(P.linear_fwd_swiglu(gd, ud, wprep, n, fmt, sp))
    xb = Q.swiglu_bf16(g, u)
    y_ref = host(P.linear_fwd_prepared(dev_bf16(xb), wprep, n, fmt, sp))
    assert np.array_equal(y.view(np.uint32), y_ref.view(np.uint32)), "fused and unfused Y differ"
    if m * d * n <= 2**31:
        o = Q.resq_forward(fmt, sp, bf16_bits_to_f32(xb), bf16_bits_to_f32(wb))
        assert_close(y, o["y64"], f"Y {fmt} {sp}")
    torch.cuda.synchronize()


def test_swiglu_rounding_edges():
    """Inputs where silu(g) * u is exactly a bf16 rounding midpoint (g = 64 or 128, where
    silu(g) = g in float64, and u = midpoint / g), g on both sides of the float32 fast path's
    limits (-80, 2^-100), tiny and huge magnitudes and signed zeros:
    the fused X must round like the oracle's, checked through Y (bit for bit against the
    unfused forward of the oracle's X)."""
    import paper_2607_26515_amd as P
    log("swiglu rounding edges")
    rng = np.random.default_rng(3)
    m, d = 64, 256
    g = rng.choice(np.array([0.0, -0.0, 64.0, 128.0, -80.0, -79.9, -80.1, -100.0, 1e-30, -1e-30,
                             2.0**-99, 2.0**-101, 3.0, 0.5, -7.25, 15.0], np.float32), (m, d))
    mids = (rng.integers(0x3000, 0x4F00, (m, d)).astype(np.uint32) << 16 | 0x8000).view(np.float32)
    tie = (g == 64.0) | (g == 128.0)
    u = np.where(tie, mids / np.where(tie, g, 1.0), rng.normal(0, 1, (m, d))).astype(np.float32)
    x64 = g.astype(np.float64) / (1.0 + np.exp(-g.astype(np.float64))) * u.astype(np.float64)
    assert (x64[tie] == mids[tie].astype(np.float64)).all(), "precondition: exact midpoints"
    gd, ud = dev_f32(g), dev_f32(u)
    wb = weights(rng_tree(4, 1)[0], 96, d)
    for fmt in FMTS:
        qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
        wprep = P.prepare_weights(qc, qs, fmt)
        for sp in ("none", "identity"):
            y = host(P.linear_fwd_swiglu(gd, ud, wprep, 96, fmt, sp))
            xb = Q.swiglu_bf16(g, u)
            y_ref = host(P.linear_fwd_prepared(dev_bf16(xb), wprep, 96, fmt, sp))
            assert np.array_equal(y.view(np.uint32), y_ref.view(np.uint32)), (fmt, sp)
