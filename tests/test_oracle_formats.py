"""Pins for the oracle's FP4 formats (CPU only).

The oracle is checked against facts fixed outside it: the E2M1 value set (golden fixture),
exhaustive sweeps over every finite bfloat16 value compared with the integer references in
``_intref`` (a different method), reconstruction-error bounds and structural properties.
"""
import os

import numpy as np
import pytest

from oracle import formats as F
from synth import bf16_bits_to_f32, f32_to_bf16_bits
import _intref as R

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_table(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                rows.append(line.split())
    return rows


# ----------------------------------------------------------------------------------------
# E2M1 / MXFP4
# ----------------------------------------------------------------------------------------
def test_e2m1_value_set_matches_golden():
    golden = {int(c): float(v) for c, v in _golden_table("e2m1_values.txt")}
    assert sorted(golden) == list(range(8))
    codes = np.arange(32, dtype=np.uint8).reshape(1, 32) & 15  # all 16 codes, twice
    vals = F.mxfp4_dequantize(codes, np.array([[127]], dtype=np.uint8))[0]
    for c in range(16):
        mag = golden[c & 7]
        assert vals[c] == (-mag if c & 8 else mag)
        assert np.signbit(vals[c]) == bool(c & 8)


def _finite_bf16_f32():
    bits = R.finite_bf16_as_f32_bits()
    return bits, bits.view(np.float32)


def test_mxfp4_exhaustive_single_element():
    """Block [v, 0, ..., 0] for every finite bf16 v: scale and code match the integer rule."""
    bits, vals = _finite_bf16_f32()
    x = np.zeros((vals.size, 32), dtype=np.float32)
    x[:, 0] = vals
    codes, scales = F.mxfp4_quantize(x)
    assert (codes[:, 1:] == 0).all()
    for i in range(0, vals.size):
        # zeros never change a block's max, so the reference only needs the non-zero entry
        c, e = R.mx_block_ref([int(bits[i])])
        assert scales[i, 0] == e, (hex(bits[i]), scales[i, 0], e)
        assert codes[i, 0] == c[0], (hex(bits[i]), codes[i, 0], c[0])


@pytest.mark.parametrize("e", [-127, -100, -3, 0, 125])
def test_mxfp4_exhaustive_sweep_against_fixed_max(e):
    """Block [6*2**e, v, 0...]: v swept over all finite bf16; compared with the integer rule."""
    bits, vals = _finite_bf16_f32()
    big = np.float32(np.ldexp(6.0, e))
    x = np.zeros((vals.size, 32), dtype=np.float32)
    x[:, 0] = big
    x[:, 1] = vals
    codes, scales = F.mxfp4_quantize(x)
    bb = R.f32_bits(float(big))
    sel = np.arange(0, vals.size, 1)
    for i in sel:
        c, sc = R.mx_block_ref([bb, int(bits[i])])
        assert scales[i, 0] == sc
        assert codes[i, 0] == c[0] and codes[i, 1] == c[1], (e, hex(bits[i]))


def test_mxfp4_reconstruction_error_and_saturation():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((512, 256)) * np.exp(rng.uniform(-20, 20, (512, 1)))).astype(np.float32)
    x = bf16_bits_to_f32(f32_to_bf16_bits(x))
    codes, scales = F.mxfp4_quantize(x)
    xh = F.mxfp4_dequantize(codes, scales)
    e = scales.astype(np.int64) - 127
    y = np.abs(x.astype(np.float64)).reshape(512, -1, 32) / np.ldexp(1.0, e)[..., None]
    # the grid step around y: 0.5 below 2, 1 in [2, 4), 2 in [4, 6]; saturation above 6
    step = np.where(y < 2, 0.5, np.where(y < 4, 1.0, 2.0))
    err = np.abs(x.astype(np.float64) - xh).reshape(512, -1, 32) / np.ldexp(1.0, e)[..., None]
    sat = y > 6
    assert (err[~sat] <= step[~sat] / 2).all()
    assert (np.abs(xh.reshape(512, -1, 32))[sat] == 6 * np.ldexp(1.0, e)[..., None].repeat(32, -1)[sat]).all()
    # every block's max element maps to magnitude code 6 (value 4) or 7 (value 6): y in [4, 8)
    mags = (codes.reshape(512, -1, 32) & 7).max(axis=-1)
    assert set(np.unique(mags)) <= {6, 7}


def test_mxfp4_zero_block_and_negative_zero():
    x = np.zeros((2, 32), dtype=np.float32)
    x[1] = -0.0
    codes, scales = F.mxfp4_quantize(x)
    assert (scales == 0).all()  # E = -127 for an all-zero block
    assert (codes[0] == 0).all() and (codes[1] == 8).all()


# ----------------------------------------------------------------------------------------
# HiF4 (reading H1-H6)
# ----------------------------------------------------------------------------------------
def test_e6m2_codes():
    v = F.e6m2_values()
    assert (np.diff(v) > 0).all()
    assert v[0] == 2.0 ** -31 and v[124] == 1.0 and v[125] == 1.25 and v[127] == 1.75
    assert v[255] == 1.75 * 2.0 ** 32


def test_s1p2_value_set():
    """S1P2 = E1M2 elements: sign and k/4, k = 0..7 (e = 0 half subnormal)."""
    vals = []
    for e in (0, 1):
        for m in range(4):
            vals.append(m / 4 if e == 0 else 1 + m / 4)
    assert np.array_equal(np.array(vals), F.S1P2_MAGNITUDES)


def test_hif4_exhaustive_single_element():
    """Block [v, 0 x 63] for every finite bf16 v, against the integer reference."""
    bits, vals = _finite_bf16_f32()
    x = np.zeros((vals.size, 64), dtype=np.float32)
    x[:, 0] = vals
    codes, meta = F.hif4_quantize(x)
    zeros = [0] * 63
    for i in range(vals.size):
        c, mt = R.hif4_block_ref([int(bits[i])] + zeros)
        assert meta[i, 0] == mt, (hex(bits[i]), hex(meta[i, 0]), hex(mt))
        assert codes[i, 0] == c[0]
    assert (codes[:, 1:] == 0).all()


def _structured_blocks(rng, nblk):
    """64-element blocks whose groups of 4 and 8 span many magnitudes (exercises all levels)."""
    base = rng.standard_normal((nblk, 64))
    g8 = np.exp2(rng.integers(-4, 1, (nblk, 8, 1)))
    g4 = np.exp2(rng.integers(-2, 1, (nblk, 8, 2, 1)))
    x = (base.reshape(nblk, 8, 2, 4) * g8[..., None] * g4).reshape(nblk, 64)
    x *= np.exp2(rng.integers(-40, 40, (nblk, 1)))
    return bf16_bits_to_f32(f32_to_bf16_bits(x.astype(np.float32)))


def _in_range(x):
    """Blocks whose max fits under the largest E6M2 scale (no saturation)."""
    return np.abs(x.astype(np.float64)).max(-1) <= 1.75 * F.e6m2_values()[255]


def test_hif4_random_blocks_match_integer_reference():
    rng = np.random.default_rng(7)
    x = _structured_blocks(rng, 3000)
    codes, meta = F.hif4_quantize(x)
    bits = x.view(np.uint32)
    for i in range(x.shape[0]):
        c, mt = R.hif4_block_ref([int(u) for u in bits[i]])
        assert meta[i, 0] == mt, i
        assert list(codes[i]) == c, i


def test_hif4_fp32_inputs_match_integer_reference():
    """Residual-like float32 inputs (24-bit mantissas), including exact midpoints."""
    rng = np.random.default_rng(11)
    x = (rng.standard_normal((800, 64)) * np.exp2(rng.integers(-30, 30, (800, 1)))).astype(np.float32)
    # plant exact midpoints k + 1/2 steps of the block's finest scale in a few blocks
    x[:100] = np.float32(1.0)
    x[:100, 1:9] = np.float32(0.125 * 3)  # 1.5 * s/4 with s1 = 1 -> a k=1/2 midpoint
    codes, meta = F.hif4_quantize(x)
    bits = x.view(np.uint32)
    for i in range(x.shape[0]):
        c, mt = R.hif4_block_ref([int(u) for u in bits[i]])
        assert meta[i, 0] == mt and list(codes[i]) == c, i


def test_hif4_levels_are_maximal_and_never_clip():
    rng = np.random.default_rng(3)
    x = _structured_blocks(rng, 4000)
    x = x[_in_range(x)].astype(np.float64)
    assert x.shape[0] > 3000
    codes, meta = F.hif4_quantize(x.astype(np.float32))
    c1, b2, b3 = F.hif4_meta_fields(meta[:, 0])
    s1 = F.e6m2_values()[c1]
    a = np.abs(x)
    a8 = a.reshape(-1, 8, 8).max(-1)
    a4 = a.reshape(-1, 16, 4).max(-1)
    # level 1 is the smallest code that does not clip
    assert (1.75 * s1 >= a.max(-1)).all()
    prev = F.e6m2_values()[np.maximum(c1 - 1, 0)]
    assert ((c1 == 0) | (1.75 * prev < a.max(-1))).all()
    # levels 2 and 3: fit with the chosen shift; a further halving would clip
    s2 = s1[:, None] * 2.0 ** -b2
    assert (a8 <= 1.75 * s2).all()
    assert ((b2 == 1) | (a8 > 1.75 * s2 / 2)).all()
    s = np.repeat(s2, 2, axis=1) * 2.0 ** -b3
    assert (a4 <= 1.75 * s).all()
    assert ((b3 == 1) | (a4 > 1.75 * s / 2)).all()


def test_hif4_reconstruction_error_half_step():
    rng = np.random.default_rng(5)
    x = _structured_blocks(rng, 2000)
    x = x[_in_range(x)]
    codes, meta = F.hif4_quantize(x)
    xh = F.hif4_dequantize(codes, meta)
    c1, b2, b3 = F.hif4_meta_fields(meta[:, 0])
    s = (F.e6m2_values()[c1][:, None] * 2.0 ** -np.repeat(b2, 2, axis=1)) * 2.0 ** -b3
    step = np.repeat(s / 4, 4, axis=1)
    assert (np.abs(x.astype(np.float64) - xh) <= step / 2).all()


def test_hif4_without_finer_levels_is_plain_e6m2_scaled_e1m2():
    """When every group of 4 holds a value near the block max, b2 = b3 = 0 and the format
    reduces to E1M2 elements under one E6M2 scale: each element is round(4|x|/s1)/4 * s1."""
    rng = np.random.default_rng(9)
    x = rng.uniform(-1, 1, (500, 64))
    x.reshape(500, 16, 4)[:, :, 0] = 1.7 * np.sign(rng.standard_normal((500, 16)))
    x = x.astype(np.float32)
    codes, meta = F.hif4_quantize(x)
    c1, b2, b3 = F.hif4_meta_fields(meta[:, 0])
    assert (b2 == 0).all() and (b3 == 0).all()
    s1 = F.e6m2_values()[c1][:, None]
    y = np.abs(x.astype(np.float64)) / s1 * 4  # s1 here is a power of two times 1.0 (no ties)
    k = np.clip(np.rint(y), 0, 7)
    assert np.array_equal(codes & 7, k.astype(np.uint8))


def test_hif4_values_are_fp6_times_e6m2():
    """Each decoded value is k * 2**-b / 4 * s1 with k * 2**(2-b) an integer <= 28 that the
    FP6 E2M3 grid {0..15, 16..30 step 2} holds exactly."""
    rng = np.random.default_rng(13)
    x = _structured_blocks(rng, 1000)
    codes, meta = F.hif4_quantize(x)
    xh = F.hif4_dequantize(codes, meta)
    c1, _, _ = F.hif4_meta_fields(meta[:, 0])
    t = np.abs(xh) / F.e6m2_values()[c1][:, None] * 16
    assert (t == np.rint(t)).all() and (t <= 28).all()
    e2m3_x8 = set(range(16)) | set(range(16, 31, 2))
    assert set(np.unique(t).astype(int)) <= e2m3_x8


def test_hif4_zero_block_is_canonical():
    codes, meta = F.hif4_quantize(np.zeros((1, 64), dtype=np.float32))
    assert meta[0, 0] == 0xFFFFFF00 and (codes == 0).all()


def test_pack_unpack_nibbles_roundtrip():
    rng = np.random.default_rng(0)
    c = rng.integers(0, 16, (3, 64)).astype(np.uint8)
    p = F.pack_nibbles(c)
    assert p.shape == (3, 32)
    assert (p[:, 0] & 15 == c[:, 0]).all() and (p[:, 0] >> 4 == c[:, 1]).all()
    assert np.array_equal(F.unpack_nibbles(p), c)
