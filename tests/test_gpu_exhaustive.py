"""Every finite bf16 value through the forward path's own quantizer (the fused activation
pass that writes MFMA fragments) and the GEMM, checked bit for bit.

With W = I (each weight row holds one 1 on the diagonal) and no residual term, output (i, j)
of Y = Q(X) Q(W)^T has exactly one non-zero product, Q(X)[i, j] * Q(W)[j, j], which is exact
in float32.  So Y shows every element of Q(X) as the GPU quantized it, scaled by the one
weight value.  The oracle's Q(X) and Q(W) give the expected Y exactly."""
import numpy as np
import pytest

from oracle import formats as F
from oracle import resq as Q
from synth import bf16_bits_to_f32, f32_to_bf16_bits
from _gpu_util import dev_bf16, host, log

pytestmark = pytest.mark.gpu

FMTS = ["mxfp4", "hif4"]


def _finite_bf16():
    b = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    return b[((b >> 7) & 0xFF) != 0xFF]  # exponent field not all ones


def _identity_forward(fmt, xbits):
    import paper_2607_26515_amd as P
    m, d = xbits.shape
    wb = f32_to_bf16_bits(np.eye(d, dtype=np.float32))
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    y = host(P.linear_fwd_prepared(dev_bf16(xbits), P.prepare_weights(qc, qs, fmt), d, fmt, "none"))
    xhat = F.dequantize(fmt, *F.quantize(fmt, bf16_bits_to_f32(xbits)))
    what = F.dequantize(fmt, *F.quantize(fmt, np.eye(d, dtype=np.float32)))
    # one exact product per output; as a sum over K it starts from +0, so a -0 product
    # gives +0 (IEEE: -0 + +0 = +0), as the oracle's matmul does
    want = (xhat * np.diag(what)[None, :]).astype(np.float32) + np.float32(0.0)
    return y, want


def _check(y, want, what):
    if not np.array_equal(y.view(np.uint32), want.view(np.uint32)):
        bad = np.argwhere(y.view(np.uint32) != want.view(np.uint32))
        i, j = bad[0]
        raise AssertionError(f"{what}: {len(bad)} outputs differ, first ({i}, {j}): {y[i, j]!r} vs {want[i, j]!r}")


@pytest.mark.parametrize("fmt", FMTS)
def test_every_bf16_value_alone_in_its_block(fmt):
    """Each finite bf16 value as the only non-zero of a block (it sets every scale level),
    in the first and in the last element of the block."""
    log(f"exhaustive single values {fmt}")
    v = _finite_bf16()
    b = F.block_size(fmt)
    x = np.zeros((v.size, 2 * b), dtype=np.uint16)
    x[:, 0] = v
    x[:, 2 * b - 1] = v
    y, want = _identity_forward(fmt, x)
    _check(y, want, "single values")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("amax", [1.0, 0.21875, 6.0, 3.0 * 2.0**20, 2.0**-60])
def test_every_bf16_value_under_a_fixed_block_max(fmt, amax):
    """A block whose maximum is fixed by element 0, with every finite bf16 value of smaller
    magnitude in a position that shares element 0's level-3 group, its level-2 group only,
    or neither (HiF4), so every element code and every level-2/3 choice is taken."""
    log(f"exhaustive under max {amax} {fmt}")
    v = _finite_bf16()
    vf = bf16_bits_to_f32(v)
    v = v[np.abs(vf) <= np.float32(amax)]
    b = F.block_size(fmt)
    x = np.zeros((v.size, b), dtype=np.uint16)
    x[:, 0] = f32_to_bf16_bits(np.array([amax], np.float32))[0]
    for pos in (1, 5, 9, b - 1):
        x[:, pos] = v
    y, want = _identity_forward(fmt, x)
    _check(y, want, f"under max {amax}")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("seed", [0, 1])
def test_backward_every_bf16_value(fmt, seed):
    """Every finite bf16 value in dY (256 x 256, a seeded permutation) through the backward's
    two quantizations of dY and its GEMMs, with X = W = I: dX = Q_n(dY) Q_n(W) has one
    product per output, Q_n(dY)[i, c] Q_n(W)[c, c], and dW = Q_m(dY)^T Q_m(X) has
    Q_m(dY)[c, j] Q_m(X)[c, c]; both exact in float32."""
    import paper_2607_26515_amd as P
    log(f"exhaustive backward {fmt} seed={seed}")
    n = 256
    v = _finite_bf16()
    flat = np.zeros(n * n, dtype=np.uint16)
    flat[: v.size] = v
    dy = np.random.default_rng(seed).permutation(flat).reshape(n, n)
    eye = f32_to_bf16_bits(np.eye(n, dtype=np.float32))
    dx, dw = P.linear_bwd(dev_bf16(dy), dev_bf16(eye), dev_bf16(eye), fmt)
    g = bf16_bits_to_f32(dy)
    i32 = np.eye(n, dtype=np.float32)
    qn_dy = F.dequantize(fmt, *F.quantize(fmt, g))               # blocks along n (rows of dY)
    qm_dy = F.dequantize(fmt, *F.quantize(fmt, g.T.copy())).T     # blocks along m (columns)
    wdiag = np.diag(F.dequantize(fmt, *F.quantize(fmt, i32)))     # Q of I, either axis
    want_dx = (qn_dy * wdiag[None, :]).astype(np.float32) + np.float32(0.0)
    want_dw = (qm_dy.T * wdiag[None, :]).astype(np.float32) + np.float32(0.0)
    _check(host(dx), want_dx, "dX")
    _check(host(dw), want_dw, "dW")
