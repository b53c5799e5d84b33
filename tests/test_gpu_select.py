"""GPU <-> oracle parity of the global residual selections (Sec. 4.3): S_50% over channels,
S^{32x64}_50% over blocks and the element-wise 50% variant.  Codes, keep masks and
channel/block masks must be bit-identical to the oracle's, ties included; the forward output
with these kinds must match the oracle's Y within the float32 tolerance."""
import numpy as np
import pytest

from oracle import formats as F
from oracle import resq as Q
from synth import WORKLOADS, activations, bf16_bits_to_f32, f32_to_bf16_bits, rng_tree, weights
from _gpu_util import assert_close, assert_codes_equal, assert_scales_equal, dev_bf16, host, log, pack_bits
from test_gpu_parity import _adversarial_bits

pytestmark = pytest.mark.gpu

FMTS = ["mxfp4", "hif4"]
GLOBAL = ["channel50", "block32x64_50", "unstructured50"]


def _check_select(fmt, sp, bits):
    import paper_2607_26515_amd as P
    m, d = bits.shape
    out = P.residual_sparsify(dev_bf16(bits), fmt, sp)
    o = Q.resq_quantize_residual(fmt, sp, bf16_bits_to_f32(bits))
    assert_codes_equal(out["qx_codes"], o["qx_codes"], "Q(X) codes")
    assert_scales_equal(fmt, out["qx_scales"], o["qx_scales"], "Q(X) scales")
    assert_scales_equal(fmt, out["qr_scales"], o["qr_scales"], "Q(dX) scales")
    keep = host(out["keep_mask"])
    want = pack_bits(o["keep"])
    if not np.array_equal(keep, want):
        bad = np.argwhere(keep != want)
        raise AssertionError(f"keep mask: {len(bad)} bytes differ, first at {bad[:5].tolist()}")
    assert_codes_equal(out["qr_codes"], o["qr_codes"], "S(Q(dX)) codes")
    if sp in ("channel50", "block32x64_50"):
        got = host(out["group_mask"])
        assert np.array_equal(got, pack_bits(o["groups"].ravel())), "channel/block mask"
    # invariant: exactly floor(count / 2) items kept
    n_items = {"channel50": d, "block32x64_50": ((m + 31) // 32) * (d // 64),
               "unstructured50": m * d}[sp]
    if sp == "unstructured50":
        kept = int(np.unpackbits(keep, bitorder="little").sum())
    else:
        kept = int(np.unpackbits(host(out["group_mask"]), bitorder="little").sum())
    assert kept == n_items // 2
    return out, o


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", GLOBAL)
@pytest.mark.parametrize("m,d", [(1, 64), (37, 512), (64, 1024), (100, 2048), (256, 2048), (33, 11008)])
def test_residual_sparsify_global(fmt, sp, m, d):
    log(f"select {fmt} {sp} {m}x{d}")
    _check_select(fmt, sp, _adversarial_bits(m, d, seed=m * 11 + d))


def _representable(fmt, m, d, rng):
    """X that the format represents exactly, so Q(dX) = 0 and every selection key is 0."""
    if fmt == "mxfp4":  # E2M1 values, a 6 in every 32-block fixes the scale at 2^0
        x = rng.choice(np.array([0, .5, 1, 1.5, 2, 3, 4, 6, -.5, -1, -3, -6], np.float32), (m, d))
        x[:, ::32] = 6.0
    else:  # k/4 values, a 1.75 in every 4-group: level-1 scale 1, no level-2/3 shifts
        x = (rng.integers(-7, 8, (m, d)) / 4.0).astype(np.float32)
        x[:, ::4] = 1.75
    return x


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", GLOBAL)
@pytest.mark.parametrize("zero", [False, True])
def test_select_all_ties(fmt, sp, zero):
    """Q(dX) = 0: every key is 0 and the lowest indices are kept."""
    log(f"select all ties {fmt} {sp} zero={zero}")
    m, d = 70, 640
    x = np.zeros((m, d), np.float32) if zero else _representable(fmt, m, d, np.random.default_rng(5))
    out, o = _check_select(fmt, sp, f32_to_bf16_bits(x))
    assert not o["r"].any(), "precondition: X is exactly representable"
    flat = (o["keep"] if sp == "unstructured50" else o["groups"]).ravel()
    assert flat[: flat.size // 2].all() and not flat[flat.size // 2:].any()


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", GLOBAL)
def test_select_repeated_rows(fmt, sp):
    """Identical rows: equal channel keys and equal element keys across rows (tie ranking)."""
    log(f"select repeated rows {fmt} {sp}")
    base = _adversarial_bits(8, 1024, seed=3)
    _check_select(fmt, sp, np.tile(base[8 - 1:8], (96, 1)))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", GLOBAL)
@pytest.mark.parametrize("linear", ["qkv", "down"])
def test_select_qwen7b_layer_m512(fmt, sp, linear):
    """The Qwen2.5-7B layer at m = 512 (activations with 0.5% outlier channels x100)."""
    from synth import workload_tensors
    wl = WORKLOADS["qwen7b_layer_m512"]
    lin = next(l for l in wl.linears if l.name == linear)
    log(f"select {fmt} {sp} qwen7b {linear} m={wl.m} d={lin.d}")
    xb, _ = workload_tensors(wl, lin, seed=0)
    _check_select(fmt, sp, xb)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", GLOBAL)
@pytest.mark.parametrize("m,d,n", [(1, 64, 1), (37, 512, 33), (100, 2048, 300), (256, 1024, 640),
                                   (70, 2048, 2560)])
def test_linear_fwd_global(fmt, sp, m, d, n):
    import paper_2607_26515_amd as P
    log(f"linear_fwd {fmt} {sp} m={m} d={d} n={n}")
    rx, rw = rng_tree(m + 2 * d + n, 2)
    xb, wb = activations(rx, m, d, 0.01, 50.0), weights(rw, n, d)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    x = dev_bf16(xb)
    y = host(P.linear_fwd(x, qc, qs, fmt, sp))
    o = Q.resq_forward(fmt, sp, bf16_bits_to_f32(xb), bf16_bits_to_f32(wb))
    assert_close(y, o["y64"], f"Y {fmt} {sp}")
    y2 = host(P.linear_fwd_prepared(x, P.prepare_weights(qc, qs, fmt), n, fmt, sp))
    assert np.array_equal(y.view(np.uint32), y2.view(np.uint32))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["channel50", "block32x64_50"])
def test_select_wide_range_channels(fmt, sp):
    """Channels whose residual magnitudes span ~2^56: their float64 sums of squares can round,
    so the GPU must reproduce the defined row-by-row order (the channel keys' sequential path)
    while the other channels take the order-free path; masks must still match the oracle."""
    log(f"select wide range {fmt} {sp}")
    m, d = 96, 256
    rng = np.random.default_rng(21)
    x = rng.standard_normal((m, d)).astype(np.float32)
    for col in (5, 70, 200):
        x[0::2, col] = 2.0 ** 28 * (1 + 2.0 ** -6)
        x[1::2, col] = -(2.0 ** -28) * (1 + 3 * 2.0 ** -7)
    x[::7, 130] = 2.0 ** 20 * 1.015625  # a channel between the two ranges
    _check_select(fmt, sp, f32_to_bf16_bits(x))


@pytest.mark.parametrize("sp", ["channel50", "unstructured50"])  # 32x64 blocks need d % 64 == 0
@pytest.mark.parametrize("m,d,n", [(45, 96, 70), (33, 160, 64), (1, 32, 5)])
def test_linear_fwd_global_mx_half_step(sp, m, d, n):
    """MXFP4 with d % 64 == 32: the last K step's second half is outside the matrix, so the
    selection must write zero operand records there (a stray scale byte would poison every
    output); m % 32 != 0 leaves padding rows in the last row tile."""
    import paper_2607_26515_amd as P
    log(f"linear_fwd mxfp4 {sp} half step m={m} d={d} n={n}")
    rx, rw = rng_tree(7 * m + d + n, 2)
    xb, wb = activations(rx, m, d, 0.05, 50.0), weights(rw, n, d)
    qc, qs = P.quantize(dev_bf16(wb), "mxfp4", axis=1)
    y = host(P.linear_fwd(dev_bf16(xb), qc, qs, "mxfp4", sp))
    o = Q.resq_forward("mxfp4", sp, bf16_bits_to_f32(xb), bf16_bits_to_f32(wb))
    assert np.isfinite(y).all()
    assert_close(y, o["y64"], f"Y mxfp4 {sp}")
