"""Pins of the oracle's mixed-precision rollout linears (Table 1: W4A16 weight-only FP4,
W16A4 activation-only FP4): brute force on tiny inputs, identity weights, representable
inputs, and the blocking axis of the quantized operand."""
import math

import numpy as np
import pytest

from oracle import formats as F
from oracle import resq as Q
from synth import activations, bf16_bits_to_f32, rng_tree, weights

FMTS = ["mxfp4", "hif4"]
C = {"mxfp4": 1.0, "hif4": 1.75}  # Q(c) = c exactly (alone in its block)


def _xw(m, d, n, seed):
    rx, rw = rng_tree(seed, 2)
    return (bf16_bits_to_f32(activations(rx, m, d, 0.05, 20.0)),
            bf16_bits_to_f32(weights(rw, n, d)))


def _triple_loop(a, b):
    """sum_k a[i, k] b[j, k], exactly summed (math.fsum), rounded to float64 once."""
    m, n = a.shape[0], b.shape[0]
    y = np.zeros((m, n))
    for i in range(m):
        for j in range(n):
            y[i, j] = math.fsum(float(a[i, k]) * float(b[j, k]) for k in range(a.shape[1]))
    return y


def _q(fmt, a):
    return F.dequantize(fmt, *F.quantize(fmt, a))


@pytest.mark.parametrize("fmt", FMTS)
def test_brute_force(fmt):
    x, w = _xw(3, 128, 5, 1)
    # the quantized operand is the weight (W4A16) or the activation (W16A4), each blocked
    # along its own rows' d axis; the other one enters as given
    want4 = _triple_loop(x, _q(fmt, w))
    want16 = _triple_loop(_q(fmt, x), w)
    np.testing.assert_allclose(Q.w4a16_forward(fmt, x, w)["y64"], want4, rtol=1e-13, atol=1e-300)
    np.testing.assert_allclose(Q.w16a4_forward(fmt, x, w)["y64"], want16, rtol=1e-13, atol=1e-300)
    assert not np.allclose(want4, want16)  # the two forms differ on outlier data


@pytest.mark.parametrize("fmt", FMTS)
def test_identity_weights(fmt):
    """W4A16 with W = c I keeps X itself (no quantization of the activations); W16A4 with
    W = I gives Q(X) itself."""
    x, _ = _xw(16, 256, 1, 2)
    d = x.shape[1]
    eye_c = np.eye(d, dtype=np.float32) * np.float32(C[fmt])
    assert np.array_equal(_q(fmt, eye_c), eye_c)
    assert np.array_equal(Q.w4a16_forward(fmt, x, eye_c)["y"], (np.float64(C[fmt]) * x).astype(np.float32))
    xhat = _q(fmt, x)
    assert not np.array_equal(xhat, x)
    assert np.array_equal(Q.w16a4_forward(fmt, x, np.eye(d, dtype=np.float32))["y"], xhat.astype(np.float32))


def _on_grid(fmt, rows, d, seed):
    """Values the format represents exactly, with every block's maximum at the top of its
    scale (MXFP4: 6 2^E; HiF4: 7/4 s1 with s1 = 2^e (1 + m/4)), so Q returns them unchanged."""
    rng = np.random.default_rng(seed)
    b = F.block_size(fmt)
    nb = d // b
    if fmt == "mxfp4":
        grid = np.array([0, .5, 1, 1.5, 2, 3, 4, 6])
        mag = grid[rng.integers(0, 8, (rows, nb, b))]
        mag[:, :, 0] = 6.0
        scale = 2.0 ** rng.integers(-8, 4, (rows, nb, 1))
    else:
        mag = rng.integers(0, 8, (rows, nb, b)) / 4.0
        mag[:, :, 0] = 1.75
        scale = 2.0 ** rng.integers(-8, 4, (rows, nb, 1)) * (1 + rng.integers(0, 4, (rows, nb, 1)) / 4)
    sign = np.where(rng.random((rows, nb, b)) < 0.5, -1.0, 1.0)
    return (sign * mag * scale).reshape(rows, d).astype(np.float32)


@pytest.mark.parametrize("fmt", FMTS)
def test_representable_operands_give_the_plain_product(fmt):
    """Quantizing an operand already on the format's grid changes nothing, so each mixed
    form is then the plain product X W^T.  (HiF4's quantizer is not idempotent in general:
    its level-1 scale is the smallest that holds the block maximum, and Q(x)'s maximum can
    need a smaller one; these inputs hold the top of their scale.)"""
    x, w = _xw(8, 256, 12, 3)
    xr, wr = _on_grid(fmt, 8, 256, 5), _on_grid(fmt, 12, 256, 6)
    assert np.array_equal(_q(fmt, xr), xr) and np.array_equal(_q(fmt, wr), wr)
    plain = lambda a, b: np.asarray(a, np.float64) @ np.asarray(b, np.float64).T
    assert np.array_equal(Q.w4a16_forward(fmt, x, wr)["y64"], plain(x, wr))
    assert np.array_equal(Q.w16a4_forward(fmt, xr, w)["y64"], plain(xr, w))


@pytest.mark.parametrize("fmt", FMTS)
def test_weight_blocks_run_along_d(fmt):
    """An outlier in one weight row leaves the other rows' quantization alone (blocks along
    d, one output feature per row): with X = I, Y = Q(W)^T row by row."""
    _, w = _xw(1, 128, 40, 4)
    w[0, 0] = np.float32(1000.0)
    y = Q.w4a16_forward(fmt, np.eye(128, dtype=np.float32), w)["y64"]
    for j in (1, 17, 39):
        assert np.array_equal(y[:, j], _q(fmt, w[j:j + 1])[0].astype(np.float64))
    assert np.count_nonzero(y[:, 1:]) > 0.5 * y[:, 1:].size
