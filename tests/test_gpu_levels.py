"""GPU <-> oracle parity of the other levels and k:g patterns of the residual sparsity
functions.  Sec. 4.3 defines S_{M:N}, S_alpha% and S^{MxN}_alpha% for any level; the paper's
experiments use 50% only and Sec. 6 leaves other levels open.  Covered here: the local S_k:4
and S_k:8 patterns applied inside the residual pass (both output layouts), and the channel,
32 x 64 block and element-wise selections at levels other than 50%.  Codes and masks must be
bit-identical to the oracle's, ties included; Y must match within the float32 tolerance."""
import numpy as np
import pytest

from oracle import resq as Q
from synth import activations, bf16_bits_to_f32, f32_to_bf16_bits, rng_tree, weights
from _gpu_util import assert_close, assert_codes_equal, assert_scales_equal, dev_bf16, host, log, pack_bits
from test_gpu_parity import _adversarial_bits
from test_gpu_select import _representable

pytestmark = pytest.mark.gpu

FMTS = ["mxfp4", "hif4"]
LOCAL = ["1:4", "3:4", "1:8", "2:8", "4:8", "7:8"]
LEVELS = ["channel25", "channel75", "block32x64_25", "block32x64_75", "unstructured10",
          "unstructured75", "unstructured99"]


def _n_items(fam, m, d):
    return {"channel": d, "block": ((m + 31) // 32) * (d // 64), "unstructured": m * d}[fam]


def _check(fmt, sp, bits):
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
    fam, par = Q.parse_sparsity(sp)
    kept_elems = np.unpackbits(keep, axis=-1, bitorder="little")[:, :d].astype(bool)
    if fam == "local":
        k, g = par
        assert (kept_elems.reshape(m, d // g, g).sum(-1) == k).all()
    else:
        if fam in ("channel", "block"):
            got = host(out["group_mask"])
            assert np.array_equal(got, pack_bits(o["groups"].ravel())), "channel/block mask"
            kept = int(np.unpackbits(got, bitorder="little").sum())
        else:
            kept = int(kept_elems.sum())
        assert kept == _n_items(fam, m, d) * par // 100
    return out, o


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", LOCAL)
@pytest.mark.parametrize("m,d", [(1, 64), (37, 512), (256, 2048), (33, 11008)])
def test_residual_sparsify_local_patterns(fmt, sp, m, d):
    log(f"residual_sparsify {fmt} {sp} {m}x{d}")
    _check(fmt, sp, _adversarial_bits(m, d, seed=m * 13 + d))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", LEVELS)
@pytest.mark.parametrize("m,d", [(1, 64), (37, 512), (100, 2048), (33, 11008)])
def test_residual_sparsify_levels(fmt, sp, m, d):
    log(f"select {fmt} {sp} {m}x{d}")
    _check(fmt, sp, _adversarial_bits(m, d, seed=m * 17 + d))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["channel25", "block32x64_75", "unstructured10"])
def test_levels_all_ties(fmt, sp):
    """Q(dX) = 0: every key is 0, so the lowest indices fill the kept count."""
    log(f"levels all ties {fmt} {sp}")
    m, d = 70, 640
    x = _representable(fmt, m, d, np.random.default_rng(6))
    out, o = _check(fmt, sp, f32_to_bf16_bits(x))
    flat = (o["keep"] if sp.startswith("unstructured") else o["groups"]).ravel()
    n = flat.sum()
    assert n > 0 and flat[:n].all() and not flat[n:].any()


def _linear(fmt, sp, m, d, n, seed, out="f32"):
    import paper_2607_26515_amd as P
    rx, rw = rng_tree(seed, 2)
    xb, wb = activations(rx, m, d, 0.01, 50.0), weights(rw, n, d)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    x = dev_bf16(xb)
    y = host(P.linear_fwd(x, qc, qs, fmt, sp))
    y2 = host(P.linear_fwd_prepared(x, P.prepare_weights(qc, qs, fmt), n, fmt, sp))
    assert np.array_equal(y.view(np.uint32), y2.view(np.uint32))
    return y, xb, wb


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", LOCAL + LEVELS)
@pytest.mark.parametrize("m,d,n", [(37, 512, 33), (100, 2048, 300), (256, 2048, 640)])
def test_linear_fwd_levels(fmt, sp, m, d, n):
    log(f"linear_fwd {fmt} {sp} m={m} d={d} n={n}")
    y, xb, wb = _linear(fmt, sp, m, d, n, seed=m + 5 * d + n)
    o = Q.resq_forward(fmt, sp, bf16_bits_to_f32(xb), bf16_bits_to_f32(wb))
    assert_close(y, o["y64"], f"Y {fmt} {sp}")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp,m,d", [("channel1", 16, 64), ("block32x64_99", 3, 64),
                                    ("unstructured1", 1, 64)])
def test_levels_that_keep_nothing(fmt, sp, m, d):
    """A kept count that rounds down to 0: S(Q(dX)) is all +0 codes and Y equals the plain
    FP4 linear (adding zero products leaves every float32 sum unchanged)."""
    log(f"levels keep nothing {fmt} {sp} {m}x{d}")
    out, o = _check(fmt, sp, _adversarial_bits(m, d, seed=d + m))
    assert not host(out["keep_mask"]).any() and not host(out["qr_codes"]).any()
    y, _, _ = _linear(fmt, sp, m, d, 96, seed=m + d)
    y0, _, _ = _linear(fmt, "none", m, d, 96, seed=m + d)
    assert np.array_equal(y, y0)
