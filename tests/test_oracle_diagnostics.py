"""Pins for the oracle's Figs. 2-4 activation statistics (CPU only)."""
import math

import numpy as np
import pytest

from oracle import diagnostics as D
from oracle import formats as F
from synth import activations, bf16_bits_to_f32, rng_tree
from test_oracle_resq import _ref_quant_rows


def _x(m, d, seed, frac=0.02, scale=50.0):
    return bf16_bits_to_f32(activations(rng_tree(seed, 1)[0], m, d, frac, scale))


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_brute_force(fmt):
    """Every statistic from explicit loops over independently quantized values."""
    m, d, b = 3, 128, F.block_size(fmt)
    x = _x(m, d, seed=21, frac=0.05)
    T = 4.0
    xq = _ref_quant_rows(fmt, x)
    r = (x.astype(np.float64) - xq).astype(np.float32)
    rq = _ref_quant_rows(fmt, r)
    want = dict(elements=m * d, zeros_x=0, zeros_qx=0, blocks=m * d // b, outlier_blocks=0)
    eq, sq, er, sr = [], [], [], []
    for i in range(m):
        for j0 in range(0, d, b):
            want["outlier_blocks"] += any(abs(float(x[i, j])) > T for j in range(j0, j0 + b))
        for j0 in range(0, d, 4):
            for vals, e_acc, s_acc in ((xq[i, j0:j0 + 4], eq, sq), (rq[i, j0:j0 + 4], er, sr)):
                order = sorted(range(4), key=lambda t: (-abs(vals[t]), t))
                for t in range(4):
                    e_acc.append(float(vals[t]) ** 2)
                    if t not in order[:2]:
                        s_acc.append(float(vals[t]) ** 2)
        want["zeros_x"] += sum(1 for v in x[i] if v == 0)
        want["zeros_qx"] += sum(1 for v in xq[i] if v == 0)
    got = D.diagnostics(fmt, x, T)
    for k in ("elements", "zeros_x", "zeros_qx", "blocks", "outlier_blocks"):
        assert got[k] == want[k], k
    for k, acc in (("energy_qx", eq), ("sse24_qx", sq), ("energy_qr", er), ("sse24_qr", sr)):
        assert got[k] == pytest.approx(math.fsum(acc), rel=1e-12), k


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_zero_input(fmt):
    x = np.zeros((5, 256), np.float32)
    x[1, 3] = -0.0
    s = D.diagnostics(fmt, x, 0.0)
    assert s["zeros_x"] == s["zeros_qx"] == 5 * 256
    assert s["outlier_blocks"] == 0
    assert s["energy_qx"] == s["sse24_qx"] == s["energy_qr"] == s["sse24_qr"] == 0.0


def test_mx_zero_collapse_closed_form():
    """One 2^10 outlier per 32-block and ones elsewhere: the shared scale 2^8 maps 1.0 to 0
    (below half of the smallest step 0.5 * 2^8), so 31 of every 32 elements collapse."""
    m, d = 4, 256
    x = np.ones((m, d), np.float32)
    x[:, ::32] = 1024.0
    s = D.diagnostics("mxfp4", x, 100.0)
    assert s["zeros_x"] == 0 and s["zeros_qx"] == m * d * 31 // 32
    assert s["outlier_blocks"] == s["blocks"] == m * d // 32
    # Q(X) keeps only the outliers: energy 1024^2 per block; S_2:4 keeps them (they lead
    # their group), so it prunes only zeros
    assert s["energy_qx"] == m * (d // 32) * 1024.0 ** 2 and s["sse24_qx"] == 0.0
    # the residual is the collapsed ones: Q(dX) = 1.0 exactly, half pruned by S_2:4
    assert s["energy_qr"] == m * d * 31 / 32
    assert s["sse24_qr"] == m * (d // 4) * 2 - m * (d // 32) * 1


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_representable_input_has_no_residual(fmt):
    rng = np.random.default_rng(3)
    if fmt == "mxfp4":
        x = rng.choice(np.array([0, .5, 1, 1.5, 2, 3, 4, 6, -.5, -1, -3, -6], np.float32), (8, 128))
        x[:, ::32] = 6.0
    else:
        x = (rng.integers(-7, 8, (8, 128)) / 4.0).astype(np.float32)
        x[:, ::4] = 1.75
    s = D.diagnostics(fmt, x, 10.0)
    assert s["energy_qr"] == s["sse24_qr"] == 0.0
    assert s["energy_qx"] == float(np.sum(x.astype(np.float64) ** 2))
    assert s["zeros_qx"] == s["zeros_x"] == int(np.count_nonzero(x == 0))


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_invariants(fmt):
    x = _x(64, 512, seed=4)
    s = D.diagnostics(fmt, x, 3.0)
    # S_2:4 prunes the two smallest of every four: at most half of each group's energy
    assert 0 < s["sse24_qx"] <= 0.5 * s["energy_qx"]
    assert 0 < s["sse24_qr"] <= 0.5 * s["energy_qr"]
    # more zeros after quantization; fewer outlier blocks at a higher threshold
    assert s["zeros_qx"] >= s["zeros_x"]
    counts = [D.diagnostics(fmt, x, t)["outlier_blocks"] for t in (0.5, 2.0, 8.0, 1e9)]
    assert counts == sorted(counts, reverse=True) and counts[-1] == 0
    # the threshold is strict: T = max|x| finds no block, the next float below finds one
    amax = np.float32(np.abs(x).max())
    assert D.diagnostics(fmt, x, float(amax))["outlier_blocks"] == 0
    assert D.diagnostics(fmt, x, float(np.nextafter(amax, np.float32(0))))["outlier_blocks"] >= 1
    mse, rmse = D.mse_rmse(s, "qr")
    assert rmse == pytest.approx(math.sqrt(mse)) and mse == s["sse24_qr"] / s["elements"]


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_residual_is_more_robust_to_2_4_on_outlier_data(fmt):
    """Sec. 4.3 (Fig. 4): S_2:4 costs Q(Delta X) a smaller MSE than Q(X) on activations with
    outlier channels (a statistical check)."""
    x = _x(128, 2048, seed=9, frac=0.01, scale=50.0)
    s = D.diagnostics(fmt, x, 10.0)
    assert D.mse_rmse(s, "qr")[0] < D.mse_rmse(s, "qx")[0]
