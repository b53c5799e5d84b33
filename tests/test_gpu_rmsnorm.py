"""GPU parity of the forward with the RMSNorm producer fused into the quantization pass
(resq_linear_fwd_prepared_rmsnorm, reading N1): per row the factor r = 1 / sqrt(mean(H^2) +
eps) from the exact sum of squares, then X = bf16(f32(f32(H r) gamma)) formed on the fly.
With X computed by the oracle and passed to the plain prepared forward, Y must be the same
bit for bit (same Q(X), dX, S and GEMM), and it must match the oracle's Y."""
import numpy as np
import pytest

from oracle import resq as Q
from synth import activations, bf16_bits_to_f32, f32_to_bf16_bits, rng_tree, weights
from _gpu_util import assert_close, dev_bf16, host, log

pytestmark = pytest.mark.gpu

FMTS = ["mxfp4", "hif4"]


def _gamma(d, seed):
    g = 1.0 + 0.3 * np.random.default_rng(seed).standard_normal(d)
    return f32_to_bf16_bits(g.astype(np.float32))


def _run(h_bits, gamma_bits, eps, fmt, sp, n, wb, layout="plain"):
    """Fused Y and the unfused Y of the oracle's X, for H given as bf16 bit patterns."""
    import torch
    import paper_2607_26515_amd as P
    m, d = h_bits.shape
    if layout == "strided":    # row stride d + 1: the kernels' 2-byte load paths
        hd = dev_bf16(np.pad(h_bits, ((0, 0), (0, 1))))[:, :d]
    else:
        hd = dev_bf16(h_bits)
    if layout == "gamma_offset":  # gamma 2 bytes past a 16-byte boundary
        gbuf = dev_bf16(np.concatenate([np.zeros(1, np.uint16), gamma_bits]))
        gd = gbuf[1:]
    else:
        gd = dev_bf16(gamma_bits)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    wprep = P.prepare_weights(qc, qs, fmt)
    y = host(P.linear_fwd_rmsnorm(hd, gd, eps, wprep, n, fmt, sp))
    xb = Q.rmsnorm_bf16(bf16_bits_to_f32(h_bits), bf16_bits_to_f32(gamma_bits), eps)
    y_ref = host(P.linear_fwd_prepared(dev_bf16(xb), wprep, n, fmt, sp))
    torch.cuda.synchronize()
    return y, y_ref, xb


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["none", "identity", "2:4", "4:8", "channel50", "block32x64_50",
                                "unstructured50"])
@pytest.mark.parametrize("m,d,n,layout", [(37, 512, 100, "plain"), (100, 2048, 300, "gamma_offset"),
                                          (256, 3584, 512, "plain"), (33, 640, 64, "strided")])
def test_rmsnorm_forward(fmt, sp, m, d, n, layout):
    log(f"rmsnorm {fmt} {sp} m={m} d={d} n={n} {layout}")
    rh, rw = rng_tree(m + d + n, 2)
    h = activations(rh, m, d, 0.01, 30.0, dist="t3")
    gamma = _gamma(d, m + n)
    wb = weights(rw, n, d)
    y, y_ref, xb = _run(h, gamma, 1e-6, fmt, sp, n, wb, layout)
    assert np.array_equal(y.view(np.uint32), y_ref.view(np.uint32)), "fused and unfused Y differ"
    if m * d * n <= 2**31:
        o = Q.resq_forward(fmt, sp, bf16_bits_to_f32(xb), bf16_bits_to_f32(wb))
        assert_close(y, o["y64"], f"Y {fmt} {sp}")


def test_rmsnorm_row_edges():
    """Rows whose statistics sit on the edges of the definition: all zeros (t = eps), one power
    of two repeated (r exact), squares summing exactly to a float32 rounding midpoint (1 +
    2^-24, to the even 1) and just past it (a further 2^-60 squared), bf16 subnormals (squares
    far below float32's range: the sum rounds to 0), values near 2^-68 (the sum is a float32
    subnormal), values near 2^64 (the sum overflows to inf, r = 0, X = +-0), an eps larger
    than the mean square, and mixed signs and signed zeros; checked through Y, bit for bit,
    against the unfused forward of the oracle's X with and without the residual term."""
    rng = np.random.default_rng(17)
    m, d, n = 64, 256, 96
    rows = []
    for i in range(m):
        kind = i % 8
        v = np.zeros(d, np.float32)
        if kind == 1:
            v[:] = 2.0 ** int(rng.integers(-40, 40)) * (-1.0) ** i
        elif kind == 2:
            v[0], v[1] = 1.0, 2.0**-12
        elif kind == 3:
            v[0], v[1], v[2] = 1.0, 2.0**-12, 2.0**-60
        elif kind == 4:
            v[:] = rng.integers(1, 128, d) * 2.0**-133 * rng.choice([-1.0, 1.0], d)
        elif kind == 5:
            v[:] = rng.normal(0, 1, d) * 2.0**64
        elif kind == 6:
            v[:] = rng.normal(0, 1, d) * 2.0**-68
        elif kind == 7:
            v[:] = rng.standard_t(3, d)
            v[::5] = -0.0
        rows.append(v)
    h = f32_to_bf16_bits(np.array(rows, np.float32))
    gamma = _gamma(d, 3)
    wb = weights(rng_tree(5, 1)[0], n, d)
    for fmt in FMTS:
        for sp in ("none", "identity", "2:4"):
            for eps in (1e-6, 2.0**-126, 0.25):
                y, y_ref, _ = _run(h, gamma, eps, fmt, sp, n, wb)
                assert np.array_equal(y.view(np.uint32), y_ref.view(np.uint32)), (fmt, sp, eps)


def test_rmsnorm_identity_weights_read_out_x():
    """With W = I (d = n = 128) and no residual term, each output is one exact product
    Q(X)_ij Q(I)_jj, so the fused path's Q(X) is compared with the oracle's quantization of
    the oracle's X bit for bit, on outlier-heavy rows."""
    from oracle import formats as F
    m, d = 96, 128
    h = activations(rng_tree(23, 1)[0], m, d, 0.05, 100.0, dist="t3")
    gamma = _gamma(d, 9)
    wb = f32_to_bf16_bits(np.eye(d, dtype=np.float32))
    for fmt in FMTS:
        y, _, xb = _run(h, gamma, 1e-6, fmt, "none", d, wb)
        qx = F.dequantize(fmt, *F.quantize(fmt, bf16_bits_to_f32(xb)))
        qi = np.diag(F.dequantize(fmt, *F.quantize(fmt, np.eye(d, dtype=np.float32))))
        # a sum over K starting from +0: a -0 product gives +0, as the oracle's matmul does
        want = (qx * qi[None, :]).astype(np.float32) + np.float32(0.0)
        assert np.array_equal(y.view(np.uint32), want.view(np.uint32)), fmt


def test_rmsnorm_largest_d():
    """d = 2^18, the largest the producer takes: a row of one value with the largest bf16
    significand (255 / 128 * 2^e) fills each per-wave bin of the square-sum histogram to
    65536 * 255^2, 99.2% of its 32-bit range; a second row mixes magnitudes, a third is
    zero.  The GEMM over K = 2^18 splits K."""
    import paper_2607_26515_amd as P
    log("rmsnorm d = 2^18")
    m, d, n = 3, 1 << 18, 32
    rng = np.random.default_rng(29)
    rows = np.zeros((m, d), np.float32)
    rows[0] = 255.0 / 128.0 * 2.0**-3
    rows[1] = rng.standard_t(3, d) * np.exp2(rng.integers(-20, 20, d))
    h = f32_to_bf16_bits(rows)
    assert (h[0] & 0x7F == 0x7F).all()
    gamma = _gamma(d, 31)
    wb = weights(rng_tree(6, 1)[0], n, d)
    assert P.gemm_plan("hif4", m, n, d, True)["ksplit"] > 1
    for fmt in FMTS:
        y, y_ref, _ = _run(h, gamma, 1e-6, fmt, "2:4", n, wb)
        assert np.array_equal(y.view(np.uint32), y_ref.view(np.uint32)), fmt
