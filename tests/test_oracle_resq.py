"""Pins for the oracle's residual, sparsity functions, GEMMs and cost model (CPU only)."""
import math
import os

import numpy as np
import pytest

from oracle import formats as F
from oracle import resq as Q
from synth import activations, bf16_bits_to_f32, f32_to_bf16_bits, rng_tree, weights
import _intref as R

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bf16(a):
    return bf16_bits_to_f32(f32_to_bf16_bits(np.asarray(a, np.float32)))


def _outlier_x(m, d, seed=0, frac=0.01, scale=50.0):
    return bf16_bits_to_f32(activations(rng_tree(seed, 1)[0], m, d, frac, scale))


# ----------------------------------------------------------------------------------------
# Eq. 2: residual
# ----------------------------------------------------------------------------------------
@pytest.mark.parametrize("fmt", F.FORMATS)
def test_residual_is_exact(fmt):
    """Q(X) + Delta X == X bit-exactly in float32, for outlier data and extreme values."""
    x = _outlier_x(64, 512)
    x[0, :64] = bf16_bits_to_f32(np.arange(1, 65, dtype=np.uint16))  # bf16 subnormals
    x[1, :64] = np.float32(3.0e9)  # large, inside the HiF4 scale range
    x[2, :] = 0.0
    x[3, ::2] = -0.0
    codes, sc = F.quantize(fmt, x)
    xh = F.dequantize(fmt, codes, sc)
    r = Q.residual(x, xh)
    assert r.dtype == np.float32
    assert np.array_equal(xh.astype(np.float32) + r, x)
    assert np.array_equal(xh + r.astype(np.float64), x.astype(np.float64))


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_representable_x_has_zero_residual(fmt):
    rng = np.random.default_rng(4)
    codes = rng.integers(0, 16, (8, 128)).astype(np.uint8)
    if fmt == "mxfp4":
        sc = rng.integers(100, 140, (8, 4)).astype(np.uint8)
        codes.reshape(8, 4, 32)[:, :, 0] = 7  # make the block max 6 * 2**e (scale is stable)
    else:
        _, sc = F.hif4_quantize(rng.standard_normal((8, 128)).astype(np.float32))
    x = F.dequantize(fmt, codes, sc).astype(np.float32)
    out = Q.resq_quantize_residual(fmt, "identity", x)
    assert np.array_equal(out["xhat"], x.astype(np.float64))
    assert (out["r"] == 0).all() and ((out["qr_codes"] & 7) == 0).all()
    w = _bf16(rng.standard_normal((5, 128)) * 0.02)
    y_resq = Q.resq_forward(fmt, "2:4", x, w)["y64"]
    y_eq1 = Q.resq_forward(fmt, "none", x, w)["y64"]
    assert np.array_equal(y_resq, y_eq1)


# ----------------------------------------------------------------------------------------
# Sec. 4.3: sparsity functions
# ----------------------------------------------------------------------------------------
def _tie_heavy(rng, m, d):
    """Values with many exact ties (small integers, random signs)."""
    return (rng.integers(0, 4, (m, d)) * rng.choice([-1.0, 1.0], (m, d))).astype(np.float64)


def test_keep_2_4_brute_force_and_invariants():
    rng = np.random.default_rng(0)
    v = _tie_heavy(rng, 37, 64)
    keep = Q.keep_2_4(v)
    assert (keep.reshape(37, 16, 4).sum(-1) == 2).all()
    for i in range(v.shape[0]):
        for g in range(16):
            grp = [(-abs(v[i, 4 * g + t]), t) for t in range(4)]
            want = {t for _, t in sorted(grp)[:2]}
            got = {t for t in range(4) if keep[i, 4 * g + t]}
            assert got == want


def _brute_top_half(keys):
    order = sorted(range(len(keys)), key=lambda i: (-keys[i], i))
    return set(order[: len(keys) // 2])


def test_channel50_brute_force_and_invariants():
    rng = np.random.default_rng(1)
    for m, d in [(5, 8), (33, 64), (7, 130)]:
        v = _tie_heavy(rng, m, d)
        keep, ch = Q.keep_channel50(v)
        assert ch.sum() == d // 2
        keys = [math.fsum(float(t) ** 2 for t in v[:, j]) for j in range(d)]
        assert set(np.nonzero(ch)[0]) == _brute_top_half(keys)
        assert (keep == ch[None, :]).all()


def test_channel_keys_are_exact_sums_on_ranged_data():
    x = _outlier_x(96, 256, seed=3)
    out = Q.resq_quantize_residual("hif4", "identity", x)
    rh = F.dequantize("hif4", out["qr_codes_dense"], out["qr_scales"])
    keys = Q.channel_keys(rh)
    for j in range(0, 256, 17):
        assert keys[j] == math.fsum(float(t) ** 2 for t in rh[:, j])


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_block50_brute_force_and_invariants(fmt):
    rng = np.random.default_rng(2)
    for m, d in [(32, 128), (70, 192), (5, 64)]:
        v = _tie_heavy(rng, m, d)
        keep, blk = Q.keep_block50(v, fmt)
        nI, nJ = (m + 31) // 32, d // 64
        assert blk.shape == (nI, nJ) and blk.sum() == (nI * nJ) // 2
        keys = []
        for I in range(nI):
            for J in range(nJ):
                keys.append(math.fsum(float(t) ** 2 for t in v[32 * I:32 * I + 32, 64 * J:64 * J + 64].ravel()))
        assert set(np.nonzero(blk.ravel())[0]) == _brute_top_half(keys)
        for I in range(nI):
            for J in range(nJ):
                assert (keep[32 * I:32 * I + 32, 64 * J:64 * J + 64] == blk[I, J]).all()


def test_unstructured50_brute_force_and_invariants():
    rng = np.random.default_rng(3)
    for m, d in [(3, 8), (9, 64), (5, 12)]:
        v = _tie_heavy(rng, m, d)
        keep = Q.keep_unstructured50(v)
        assert keep.sum() == (m * d) // 2
        flat = [abs(t) for t in v.ravel()]
        assert set(np.nonzero(keep.ravel())[0]) == _brute_top_half(flat)


@pytest.mark.parametrize("k,g", [(1, 4), (3, 4), (1, 8), (2, 8), (4, 8), (7, 8)])
def test_keep_k_of_g_brute_force_and_invariants(k, g):
    """S_{k:g} (Sec. 4.3 defines S_{M:N} for any M, N): the k largest |value| of every g, ties
    to the lower index, by sorting each group."""
    rng = np.random.default_rng(10 + 8 * k + g)
    m, d = 13, 64
    v = _tie_heavy(rng, m, d)
    keep = Q.keep_k_of_g(v, k, g)
    assert (keep.reshape(m, d // g, g).sum(-1) == k).all()
    for i in range(m):
        for q in range(d // g):
            grp = [(-abs(v[i, g * q + t]), t) for t in range(g)]
            want = {t for _, t in sorted(grp)[:k]}
            assert {t for t in range(g) if keep[i, g * q + t]} == want


def _brute_top(keys, pct):
    order = sorted(range(len(keys)), key=lambda i: (-keys[i], i))
    return set(order[: len(keys) * pct // 100])


@pytest.mark.parametrize("pct", [1, 25, 30, 75, 99])
def test_global_levels_brute_force_and_nesting(pct):
    """S_alpha% over channels, 32 x 64 blocks and elements for alpha != 50: floor(count *
    alpha / 100) kept by a full sort; a higher level keeps a superset."""
    rng = np.random.default_rng(pct)
    m, d = 70, 192
    v = _tie_heavy(rng, m, d)
    keep, ch = Q.keep_channel(v, pct)
    keys = [math.fsum(float(t) ** 2 for t in v[:, j]) for j in range(d)]
    assert set(np.nonzero(ch)[0]) == _brute_top(keys, pct) and ch.sum() == d * pct // 100
    assert (keep == ch[None, :]).all()
    keep, blk = Q.keep_block(v, "hif4", pct)
    nI, nJ = (m + 31) // 32, d // 64
    bkeys = [math.fsum(float(t) ** 2 for t in v[32 * I:32 * I + 32, 64 * J:64 * J + 64].ravel())
             for I in range(nI) for J in range(nJ)]
    assert set(np.nonzero(blk.ravel())[0]) == _brute_top(bkeys, pct)
    keep = Q.keep_unstructured(v, pct)
    flat = [abs(t) for t in v.ravel()]
    assert set(np.nonzero(keep.ravel())[0]) == _brute_top(flat, pct)
    if pct < 99:
        assert (Q.keep_unstructured(v, pct) <= Q.keep_unstructured(v, pct + 1)).all()
        assert (Q.keep_channel(v, pct)[1] <= Q.keep_channel(v, pct + 1)[1]).all()


def test_levels_that_round_to_zero_keep_nothing():
    v = _tie_heavy(np.random.default_rng(4), 3, 64)
    assert not Q.keep_channel(v, 1)[1].any()          # floor(64 / 100) = 0
    assert not Q.keep_block(v, "mxfp4", 99)[1].any()  # one block: floor(99 / 100) = 0
    assert Q.keep_unstructured(v, 1).sum() == 1       # floor(192 / 100) = 1: the largest |value|


def test_sparsity_names():
    assert Q.parse_sparsity("2:4") == ("local", (2, 4))
    assert Q.parse_sparsity("4:8") == ("local", (4, 8))
    assert Q.parse_sparsity("channel25") == ("channel", 25)
    assert Q.parse_sparsity("block32x64_75") == ("block", 75)
    assert Q.parse_sparsity("unstructured50") == ("unstructured", 50)
    for bad in ("0:4", "4:4", "2:6", "channel0", "channel100", "block64x64_50", "dense"):
        with pytest.raises(ValueError):
            Q.parse_sparsity(bad)
    assert Q.flops_resq(2, 8, 4, "1:4") == 2 * 2 * 8 * 4 + 2 * 8 * 4 // 2
    assert Q.flops_resq(2, 8, 4, "unstructured75") == 2 * 2 * 8 * 4 + 3 * 2 * 8 * 4 // 2


@pytest.mark.parametrize("fmt", F.FORMATS)
@pytest.mark.parametrize("sp", ["2:4", "channel50", "block32x64_50", "unstructured50", "1:4",
                                "4:8", "channel25", "block32x64_75", "unstructured30"])
def test_sparsify_zeroes_pruned_codes_and_keeps_scales(fmt, sp):
    x = _outlier_x(64, 256, seed=5)
    out = Q.resq_quantize_residual(fmt, sp, x)
    dense, kept, keep = out["qr_codes_dense"], out["qr_codes"], out["keep"]
    assert (kept[~keep] == 0).all()
    assert np.array_equal(kept[keep], dense[keep])
    assert abs(keep.mean() - Q.kept_fraction(sp)) < 0.02


# ----------------------------------------------------------------------------------------
# Eq. 1 / Eq. 3 / Eq. 4 and the backward GEMMs: brute force with independently quantized
# operands (integer reference quantizers, explicit loops over blocks along the right axis)
# ----------------------------------------------------------------------------------------
def _ref_quant_rows(fmt, x):
    """Dequantized values of x quantized along its rows, using the integer references."""
    b = F.block_size(fmt)
    ref = R.mx_block_ref if fmt == "mxfp4" else R.hif4_block_ref
    out = np.zeros(x.shape, dtype=np.float64)
    bits = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    for i in range(x.shape[0]):
        for j0 in range(0, x.shape[1], b):
            codes, sc = ref([int(u) for u in bits[i, j0:j0 + b]])
            c = np.array(codes, dtype=np.uint8)[None, :]
            s = np.array([[sc]], dtype=np.uint8 if fmt == "mxfp4" else np.uint32)
            out[i, j0:j0 + b] = F.dequantize(fmt, c, s)[0]
    return out


def _dot(a, b):
    return math.fsum(float(p) * float(q) for p, q in zip(a, b))


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_forward_brute_force(fmt):
    m, d, n = 5, 128, 3
    x = _outlier_x(m, d, seed=6, frac=0.05)
    w = bf16_bits_to_f32(weights(rng_tree(7, 1)[0], n, d))
    xq = _ref_quant_rows(fmt, x)
    wq = _ref_quant_rows(fmt, w)
    r = (x.astype(np.float64) - xq).astype(np.float32)
    rq = _ref_quant_rows(fmt, r)
    keep = Q.keep_2_4(rq)
    srq = np.where(keep, rq, 0.0)
    for sp, extra in [("none", None), ("identity", rq), ("2:4", srq)]:
        y = Q.resq_forward(fmt, sp, x, w)["y64"]
        for i in range(m):
            for j in range(n):
                want = _dot(xq[i], wq[j]) + (0.0 if extra is None else _dot(extra[i], wq[j]))
                assert y[i, j] == pytest.approx(want, rel=1e-13, abs=1e-300)


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_identity_equals_sum_of_operands(fmt):
    x = _outlier_x(33, 256, seed=8)
    w = bf16_bits_to_f32(weights(rng_tree(9, 1)[0], 17, 256))
    o = Q.resq_forward(fmt, "identity", x, w)
    rh = F.dequantize(fmt, o["qr_codes_dense"], o["qr_scales"])
    np.testing.assert_allclose(o["y64"], (o["xhat"] + rh) @ o["what"].T, rtol=1e-13, atol=1e-300)


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_backward_brute_force(fmt):
    b = F.block_size(fmt)
    m, n, d = 2 * b, b, 3
    rng = rng_tree(10, 3)
    x = bf16_bits_to_f32(activations(rng[0], m, d, 0.0, 1.0))
    w = bf16_bits_to_f32(weights(rng[1], n, d))
    dy = _bf16(rng[2].standard_normal((m, n)) * 1e-3)
    out = Q.resq_backward(fmt, dy, x, w)
    dyn = _ref_quant_rows(fmt, dy)              # blocks along n
    wn = _ref_quant_rows(fmt, w.T).T            # blocks along n (columns of W)
    dym = _ref_quant_rows(fmt, dy.T).T          # blocks along m (columns of dY)
    xm = _ref_quant_rows(fmt, x.T).T            # blocks along m (columns of X)
    for i in range(m):
        for j in range(d):
            assert out["dx64"][i, j] == pytest.approx(_dot(dyn[i], wn[:, j]), rel=1e-13, abs=1e-300)
    for k in range(n):
        for j in range(d):
            assert out["dw64"][k, j] == pytest.approx(_dot(dym[:, k], xm[:, j]), rel=1e-13, abs=1e-300)
    assert out["dx"].dtype == np.float32 and out["dw"].dtype == np.float32


# ----------------------------------------------------------------------------------------
# the paper's qualitative claims, on synthetic outlier data (statistical, not parity)
# ----------------------------------------------------------------------------------------
@pytest.mark.parametrize("fmt", F.FORMATS)
def test_resq_reduces_activation_error(fmt):
    """Sec. 4.3: the residual recovers precision lost to activation quantization."""
    x = _outlier_x(64, 1024, seed=11)
    w = bf16_bits_to_f32(weights(rng_tree(12, 1)[0], 64, 1024))
    base = Q.resq_forward(fmt, "none", x, w)
    ref = x.astype(np.float64) @ base["what"].T  # isolates the activation-side error
    err = {sp: np.linalg.norm(Q.resq_forward(fmt, sp, x, w)["y64"] - ref)
           for sp in ["none", "identity", "2:4", "channel50", "block32x64_50", "unstructured50"]}
    for sp in ["identity", "2:4", "channel50", "block32x64_50", "unstructured50"]:
        assert err[sp] < err["none"], (sp, err)
    assert err["identity"] <= min(err[s] for s in ["2:4", "channel50", "block32x64_50"])


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_residual_more_robust_to_2_4_than_activation(fmt):
    """Fig. 4: S_2:4 costs Q(Delta X) less error than it costs Q(X)."""
    x = _outlier_x(128, 1024, seed=13)
    o = Q.resq_quantize_residual(fmt, "identity", x)
    rh = F.dequantize(fmt, o["qr_codes_dense"], o["qr_scales"])
    xh = o["xhat"]
    mse_r = np.mean((rh - np.where(Q.keep_2_4(rh), rh, 0)) ** 2)
    mse_x = np.mean((xh - np.where(Q.keep_2_4(xh), xh, 0)) ** 2)
    assert mse_r < mse_x


@pytest.mark.parametrize("fmt", F.FORMATS)
def test_outliers_cause_zero_collapse(fmt):
    """Fig. 2 / Sec. 4.2: outlier channels raise the fraction of zero codes after Q."""
    clean = _outlier_x(64, 2048, seed=14, frac=0.0)
    dirty = _outlier_x(64, 2048, seed=14, frac=0.01, scale=100.0)
    z = lambda x: np.mean((F.quantize(fmt, x)[0] & 7) == 0)
    assert z(dirty) > z(clean) + 0.05


# ----------------------------------------------------------------------------------------
# Sec. 5.4: overhead cost model
# ----------------------------------------------------------------------------------------
def test_overhead_model_matches_golden():
    g = {}
    with open(os.path.join(GOLDEN, "overhead_sec5_4.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                k, v = line.split()
                g[k] = float(v)
    m, d, n = 3, 5, 7
    mdn = m * d * n
    assert Q.flops_dense(m, d, n) == g["dense_fp16_flops"] * mdn
    assert Q.flops_resq(m, d, n, "2:4") - Q.flops_dense(m, d, n) == g["resq_2_4_sparse_residual_flops"] * mdn
    assert Q.effective_cost(m, d, n, "identity", g["fp4_throughput_advantage"]) == g["effective_resq_dense_total"] * mdn
    assert Q.effective_cost(m, d, n, "2:4", g["fp4_throughput_advantage"]) == g["effective_resq_2_4_total"] * mdn
    assert Q.effective_cost(m, d, n, "none") == g["effective_dense_fp4_gemm"] * mdn
    assert Q.speedup_vs_fp16("identity") == g["speedup_resq_dense_vs_fp16"]
    assert Q.speedup_vs_fp16("2:4") == pytest.approx(g["speedup_resq_2_4_vs_fp16"], abs=1e-4)


# ----------------------------------------------------------------------------------------
# Optional bf16 output: the float32 result rounded to bf16, nearest, ties to even
# ----------------------------------------------------------------------------------------
def _bf16_nearest_exact(v32: np.float32) -> int:
    """Nearest bf16 by exact rational distance to the two bf16 values around v (ties: even)."""
    from fractions import Fraction
    u = int(np.float32(v32).view(np.uint32))
    lo = u & 0xFFFF0000
    cands = [lo >> 16, (lo >> 16) + 1]
    vals = [Fraction(float(np.uint32(c << 16).view(np.float32))) for c in cands]
    x = Fraction(float(v32))
    d = [abs(x - c) for c in vals]
    if d[0] != d[1]:
        return cands[0] if d[0] < d[1] else cands[1]
    return cands[0] if cands[0] % 2 == 0 else cands[1]


def test_round_to_bf16_special_values():
    one = 0x3F80
    cases = [(1.0, one), (1.0 + 2.0**-8, one), (1.0 + 3 * 2.0**-8, 0x3F82),
             (1.0 + 2.0**-8 + 2.0**-20, 0x3F81), (-(1.0 + 3 * 2.0**-8), 0xBF82),
             (0.0, 0), (-0.0, 0x8000), (2.0**-149, 0), (1.5 * 2.0**-133, 0x0002), (3 * 2.0**-133, 0x0003)]
    x = np.array([c[0] for c in cases], dtype=np.float32)
    got = Q.round_to_bf16(x)
    assert [int(g) for g in got] == [c[1] for c in cases]
    # values that are already bf16 are kept bit for bit
    b = R.finite_bf16_as_f32_bits()
    assert np.array_equal(Q.round_to_bf16(b.view(np.float32)), (b >> 16).astype(np.uint16))


def test_round_to_bf16_exact_distance_and_torch():
    import torch
    rng = np.random.default_rng(11)
    u = rng.integers(0, 0x7F7F0000, size=4000, dtype=np.uint64).astype(np.uint32)
    # half of them forced onto a tie or next to it
    u[:1000] = (u[:1000] & 0xFFFF0000) | 0x8000
    u[1000:1500] = (u[1000:1500] & 0xFFFF0000) | 0x7FFF
    u[1500:2000] = (u[1500:2000] & 0xFFFF0000) | 0x8001
    u[2000:3000] |= 0x80000000
    v = u.view(np.float32)
    got = Q.round_to_bf16(v)
    for k in range(0, len(v), 7):
        assert int(got[k]) == _bf16_nearest_exact(v[k]), hex(int(u[k]))
    t = torch.from_numpy(v.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, t)


# ----------------------------------------------------------------------------------------
# Fused producer of the down projection's input: X = silu(G) * U rounded once to bf16
# ----------------------------------------------------------------------------------------
def _bf16_nearest_f64_exact(v: float) -> int:
    """Nearest bf16 to a float64 by exact rational distance over the bf16 grid (ties: even)."""
    from fractions import Fraction
    x = Fraction(v)
    best = None
    lo = int(np.float32(v).view(np.uint32)) >> 16  # a bf16 near v: search its neighbours
    for c in range(max(lo - 2, 0) if v >= 0 else lo - 2, lo + 3):
        c &= 0xFFFF
        f = np.uint32(c << 16).view(np.float32)
        if not np.isfinite(f):
            continue
        dist = abs(x - Fraction(float(f)))
        key = (dist, c & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def test_round_f64_to_bf16_exact_distance():
    rng = np.random.default_rng(12)
    b = rng.integers(0x0001, 0x7F7F, size=600).astype(np.uint32)
    mids = (b << 16 | 0x8000).view(np.float32).astype(np.float64)  # exact bf16 midpoints
    ulp = np.spacing(mids)
    v = np.concatenate([mids, mids + ulp, mids - ulp, rng.normal(0, 1, 300) * 10.0 ** rng.integers(-30, 30, 300)])
    v = np.concatenate([v, -v[::3]])
    got = Q.round_f64_to_bf16(v)
    for k in range(0, len(v), 3):
        assert int(got[k]) == _bf16_nearest_f64_exact(float(v[k])), (v[k], hex(int(got[k])))
    # a float32 value is rounded once either way
    f = rng.normal(0, 1, 2000).astype(np.float32) * np.float32(3.0)
    assert np.array_equal(Q.round_f64_to_bf16(f.astype(np.float64)), Q.round_to_bf16(f))
    # ties go to even, in the subnormal range too
    assert int(Q.round_f64_to_bf16(np.array([1.0 + 2.0**-8]))[0]) == 0x3F80
    assert int(Q.round_f64_to_bf16(np.array([1.5 * 2.0**-133]))[0]) == 0x0002
    assert int(Q.round_f64_to_bf16(np.array([-2.5 * 2.0**-133]))[0]) == 0x8002


def test_swiglu_matches_library_sigmoid():
    """silu(g) * u against scipy's logistic function (an independent implementation); the two
    float64 values may differ in the last bits, which can move the bf16 result only when the
    value sits on a rounding midpoint."""
    from scipy.special import expit
    rng = np.random.default_rng(13)
    g = bf16_bits_to_f32(f32_to_bf16_bits(rng.normal(0, 3, 20000).astype(np.float32))).astype(np.float64)
    u = bf16_bits_to_f32(f32_to_bf16_bits(rng.normal(0, 2, 20000).astype(np.float32))).astype(np.float64)
    ref = g * expit(g) * u
    got = Q.swiglu_bf16(g, u)
    want = Q.round_f64_to_bf16(ref)
    diff = np.nonzero(got != want)[0]
    for k in diff:
        step = np.exp2(np.floor(np.log2(abs(ref[k]))) - 7)
        frac = abs(ref[k]) / step - np.floor(abs(ref[k]) / step)
        assert abs(frac - 0.5) < 1e-9, (g[k], u[k])
    assert len(diff) <= 2
    # closed forms: silu(0) = 0; u = 0 gives a zero; silu(g) -> g for large g
    z = Q.swiglu_bf16(np.array([0.0, 3.0, 80.0]), np.array([5.0, 0.0, 1.0]))
    assert bf16_bits_to_f32(z[:2]).tolist() == [0.0, 0.0] and bf16_bits_to_f32(z[2:]).tolist() == [80.0]


# ----------------------------------------------------------------------------------------
# Reading N1: the fused RMSNorm producer of the qkv and gate/up projections
# ----------------------------------------------------------------------------------------
def _nearest_f32_brute(v):
    """The float32 nearest to the rational v >= 0, ties to the even significand: the three
    float32 values around float(v) compared exactly as fractions."""
    from fractions import Fraction
    c = np.float32(float(v))
    cands = [np.nextafter(c, np.float32(-np.inf)), c, np.nextafter(c, np.float32(np.inf))]
    cands = [x for x in cands if np.isfinite(x) and x >= 0]
    best = min(abs(Fraction(float(x)) - v) for x in cands)
    near = [x for x in cands if abs(Fraction(float(x)) - v) == best]
    return min(near, key=lambda x: int(np.array(x, np.float32).view(np.uint32)) & 1)


def test_rmsnorm_square_sums_brute_force():
    """The exact-then-rounded sums of squares against Fraction arithmetic and a brute-force
    nearest float32, on rows that mix magnitudes 2^-133 (bf16 subnormals) to 2^60, zeros and
    signs, so that the exact sums carry far more bits than float64 holds."""
    from fractions import Fraction
    rng = np.random.default_rng(21)
    rows = []
    for i in range(60):
        d = int(rng.integers(1, 40))
        e = rng.integers(-133 if i % 3 == 0 else -30, 61 if i % 3 == 1 else 8, d)
        v = rng.integers(1, 256, d) * np.exp2(e.astype(np.float64) - 7) * rng.choice([-1, 1], d)
        v[rng.random(d) < 0.2] = 0.0
        rows.append(_bf16(v.astype(np.float32)))
    for r in rows:
        got = Q.exact_square_sums_f32(r[None, :])[0]
        want = _nearest_f32_brute(sum(Fraction(float(x)) ** 2 for x in r))
        assert got == want and np.array(got).view(np.uint32) == np.array(want).view(np.uint32), r


def test_rmsnorm_square_sum_rounding_cases():
    """Ties and the ends of the float32 range: 1 + 2^-24 is halfway between 1 and its successor
    and goes to the even 1; a further 2^-120 tips it up; 3 * 2^-13 squared is 1.125 units of
    the last place; sums below half of 2^-149 vanish, those at 2^-149 survive as subnormals;
    2^129 overflows to inf."""
    cases = [([1.0, 2.0**-12], 1.0), ([1.0, 2.0**-12, 2.0**-60], 1.0 + 2.0**-23),
             ([1.0, 3 * 2.0**-13], 1.0 + 2.0**-23), ([2.0**-75, 2.0**-75], 2.0**-149),
             ([2.0**-76, 2.0**-76, 2.0**-76], 0.0), ([2.0**-75, 2.0**-76], 2.0**-149),
             ([2.0**64, 2.0**64], np.inf), ([0.0, -0.0], 0.0), ([-3.0, 4.0], 25.0)]
    for row, want in cases:
        got = Q.exact_square_sums_f32(np.array([row], np.float32))[0]
        assert got == np.float32(want), (row, got, want)


def test_rmsnorm_constant_rows_give_gamma():
    """A row of one power of two +-2^k (d a power of two) has mean square 4^k; with eps far
    below its last place t = 4^k, q = 2^k and r = 2^-k exactly, so X = +-gamma bit for bit."""
    d = 128
    gamma = _bf16(np.random.default_rng(5).normal(0, 1, d).astype(np.float32))
    ks = [-40, -7, 0, 3, 40]
    h = np.array([[(-1.0) ** i * 2.0**k] * d for i, k in enumerate(ks)], np.float32)
    x = bf16_bits_to_f32(Q.rmsnorm_bf16(h, gamma, 2.0**-126))
    for i in range(len(ks)):
        assert np.array_equal(x[i], gamma * np.float32((-1.0) ** i)), ks[i]


def test_rmsnorm_is_scale_free():
    """Scaling H by 2^j scales s, mu and t by 4^j and r by 2^-j exactly (eps below the last
    place of mu), so X does not change."""
    rng = np.random.default_rng(6)
    h = _bf16(rng.normal(0, 1, (8, 300)).astype(np.float32))
    gamma = _bf16(rng.normal(1, 0.2, 300).astype(np.float32))
    x0 = Q.rmsnorm_bf16(h, gamma, 2.0**-126)
    for j in (-20, -3, 5, 30):
        assert np.array_equal(Q.rmsnorm_bf16(h * np.float32(2.0**j), gamma, 2.0**-126), x0), j


def test_rmsnorm_close_to_the_real_value():
    """X against a float64 evaluation of H gamma / sqrt(mean(H^2) + eps) (math.fsum for the
    mean): within half a bf16 place plus the float32 steps' few units of 2^-24, with eps
    comparable to the mean square on half the rows (a dropped eps, a mean over d - 1, a
    missing square root or a gain taken from the wrong column would all exceed it)."""
    import math
    rng = np.random.default_rng(7)
    m, d = 24, 40
    h = _bf16((rng.normal(0, 1, (m, d)) * np.exp2(rng.integers(-4, 4, (m, 1)))).astype(np.float32))
    gamma = _bf16(rng.normal(1, 0.5, d).astype(np.float32))
    for eps in (1e-6, 0.7):
        x = bf16_bits_to_f32(Q.rmsnorm_bf16(h, gamma, eps)).astype(np.float64)
        for i in range(m):
            ms = math.fsum(float(v) ** 2 for v in h[i]) / d
            ref = h[i].astype(np.float64) * gamma.astype(np.float64) / math.sqrt(ms + float(np.float32(eps)))
            half_place = np.exp2(np.floor(np.log2(np.abs(ref))) - 8)  # half a bf16 place
            tol = half_place + np.abs(ref) * 2.0**-20
            assert (np.abs(x[i] - ref) <= tol).all(), (eps, i)
