"""GPU <-> oracle parity of the Figs. 2-4 activation statistics (resq_diagnostics): counts
bit-exact, float64 sums of squares within the rounding bound of two summation orders."""
import numpy as np
import pytest

from oracle import diagnostics as D
from synth import WORKLOADS, activations, bf16_bits_to_f32, f32_to_bf16_bits, rng_tree
from _gpu_util import dev_bf16, host, log
from test_gpu_parity import _adversarial_bits

pytestmark = pytest.mark.gpu

FMTS = ["mxfp4", "hif4"]
COUNTS = ("elements", "zeros_x", "zeros_qx", "blocks", "outlier_blocks")
SUMS = ("energy_qx", "sse24_qx", "energy_qr", "sse24_qr")


def _check(fmt, bits, thr, x_dev=None):
    import paper_2607_26515_amd as P
    got = host(P.diagnostics(dev_bf16(bits) if x_dev is None else x_dev, fmt, thr))
    want = D.diagnostics(fmt, bf16_bits_to_f32(bits), thr)
    g = dict(zip(P.DIAG_STATS, got.tolist()))
    for k in COUNTS:
        assert g[k] == want[k], (k, g[k], want[k])
    # n non-negative exact terms summed in two different orders: each result is within
    # n * 2^-53 (relative) of the exact sum
    tol = 2.0 * max(bits.size, 1) * 2.0**-53
    for k in SUMS:
        assert abs(g[k] - want[k]) <= tol * want[k], (k, g[k], want[k])
    return g, want


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("m,d", [(1, 64), (37, 512), (256, 2048), (700, 2048), (33, 11008)])
def test_diagnostics_matches_oracle(fmt, m, d):
    log(f"diagnostics {fmt} {m}x{d}")
    xb = activations(rng_tree(m + d, 1)[0], m, d, 0.01, 50.0)
    _check(fmt, xb, 8.0)


@pytest.mark.parametrize("fmt", FMTS)
def test_diagnostics_adversarial_values(fmt):
    """Extreme exponents, signed zeros, rounding ties (the quantizer parity inputs)."""
    log(f"diagnostics adversarial {fmt}")
    _check(fmt, _adversarial_bits(96, 1024, seed=31), 1.0)


@pytest.mark.parametrize("fmt", FMTS)
def test_diagnostics_threshold_is_strict(fmt):
    log(f"diagnostics threshold {fmt}")
    xb = activations(rng_tree(5, 1)[0], 64, 512, 0.01, 50.0)
    amax = np.float32(np.abs(bf16_bits_to_f32(xb)).max())
    g, _ = _check(fmt, xb, float(amax))
    assert g["outlier_blocks"] == 0
    g, _ = _check(fmt, xb, float(np.nextafter(amax, np.float32(0))))
    assert g["outlier_blocks"] >= 1


def test_diagnostics_zero_collapse():
    log("diagnostics zero collapse")
    x = np.ones((40, 256), np.float32)
    x[:, ::32] = 1024.0
    g, _ = _check("mxfp4", f32_to_bf16_bits(x), 100.0)
    assert g["zeros_qx"] == 40 * 256 * 31 // 32


@pytest.mark.parametrize("fmt", FMTS)
def test_diagnostics_strided_and_unaligned_rows(fmt):
    """Row stride ldx = d + 3 (rows not 8-byte aligned: the scalar load path)."""
    import torch
    log(f"diagnostics strided {fmt}")
    m, d = 50, 640
    wide = activations(rng_tree(77, 1)[0], m, d + 3, 0.02, 30.0)
    xd = torch.from_numpy(wide.view(np.int16)).cuda()[:, :d]
    _check(fmt, np.ascontiguousarray(wide[:, :d]), 4.0, x_dev=xd)


@pytest.mark.parametrize("fmt", FMTS)
def test_diagnostics_empty_and_deterministic(fmt):
    import torch
    import paper_2607_26515_amd as P
    log(f"diagnostics empty/determinism {fmt}")
    e = host(P.diagnostics(torch.empty((0, 64), dtype=torch.int16, device="cuda"), fmt, 1.0))
    assert not e.any()
    xb = activations(rng_tree(8, 1)[0], 512, 3584, 0.005, 100.0)
    a = host(P.diagnostics(dev_bf16(xb), fmt, 10.0))
    b = host(P.diagnostics(dev_bf16(xb), fmt, 10.0))
    assert np.array_equal(a.view(np.uint64), b.view(np.uint64))


@pytest.mark.parametrize("fmt", FMTS)
def test_diagnostics_qwen7b_layer_inputs(fmt):
    """The Qwen2.5-7B block's activations at m = 512 (qkv and down inputs)."""
    from synth import workload_tensors
    wl = WORKLOADS["qwen7b_layer_m512"]
    for lin in wl.linears:
        if lin.name not in ("qkv", "down"):
            continue
        log(f"diagnostics qwen7b {fmt} {lin.name} m={wl.m} d={lin.d}")
        xb, _ = workload_tensors(wl, lin, seed=0)
        _check(fmt, xb, 10.0)
