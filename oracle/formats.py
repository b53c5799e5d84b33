"""Block-scaled FP4 formats: MXFP4 and HiF4 (oracle; test infrastructure only).

Paper Sec. 3 ("Block-Scaled Quantization") names the two formats used as Q:

* MXFP4: blocks of 32 elements, one shared E8M0 scale per block, E2M1 elements.  The paper
  cites the OCP Microscaling format; its conversion rule is used here (shared exponent =
  floor(log2(max|x|)) - 2, where 2 is the largest E2M1 exponent, clamped to the E8M0 range;
  elements rounded to nearest, ties to even, saturating at +-6).
* HiF4: blocks of 64 elements with three scale levels, an E6M2 first-level scale, one-bit
  (E1) second- and third-level scales, and S1P2 (= E1M2) elements.

The paper does not spell out HiF4's group sizes, the meaning of an E1 scale, the E6M2 bias or
the scale-selection rule.  This module implements the following reading (each point is also
listed among the readings of the paper in the design notes):

  H1  level-2 groups of 8 elements (8 per block), level-3 groups of 4 (16 per block):
      8 + 8 + 16 = 32 metadata bits per 64 elements.
  H2  an E1 scale bit b multiplies the level above it by 2**-b (finer grid for small groups).
  H3  an S1P2 element is a sign and a 3-bit magnitude k, value k/4, k = 0..7
      (E1M2 with a subnormal e=0 half: {0, .25, ..., 1.75}).
  H4  E6M2 is unsigned, value 2**(e-31) * (1 + m/4) for code 4e+m, all 256 codes finite.
  H5  level 1: the smallest E6M2 value s1 with 1.75*s1 >= max|x| (no clipping; the largest
      code when none suffices).  Levels 2 and 3: take the finer scale (bit = 1) exactly when
      the group's max|x| still fits, i.e. max|x_g| <= 1.75 * (scale above) / 2.
  H6  elements: nearest grid point, ties to the even code, saturating.

Codes: one element per array entry (a nibble, bit 3 = sign copied from x, so -0 stays -0).
Packing two nibbles per byte is a layout step done by the callers that compare with the GPU.
HiF4 metadata: one uint32 per 64-block, bits 0-7 the E6M2 code, bit 8+g the level-2 bit of
group g (g = 0..7), bit 16+h the level-3 bit of group h (h = 0..15).
"""
from __future__ import annotations

import numpy as np

MX_BLOCK = 32
HIF4_BLOCK = 64

# E2M1 magnitudes indexed by the 3-bit code (exponent bits 2..1, mantissa bit 0)
E2M1_MAGNITUDES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)
# S1P2 (= E1M2) magnitudes k/4
S1P2_MAGNITUDES = np.arange(8, dtype=np.float64) / 4.0
E8M0_BIAS = 127
E6M2_BIAS = 31


def e6m2_values() -> np.ndarray:
    """Value of every E6M2 code 0..255 (reading H4), increasing with the code."""
    c = np.arange(256)
    return np.ldexp(1.0 + (c & 3) / 4.0, (c >> 2) - E6M2_BIAS)


def _nearest_ties_even(y: np.ndarray, grid: np.ndarray) -> np.ndarray:
    """Index of the grid point nearest to y >= 0; on a tie the even index wins.

    ``grid`` is increasing along its last axis.  Values at or above the largest grid point
    saturate to it.  Below that, distances are formed in float64 and the subtraction is exact
    (y has at most 24 significant bits, the grid points at most 6 at a nearby exponent, and a
    tiny y is exactly its own distance to the zero point), so ties are detected exactly.
    """
    dist = np.abs(y[..., None] - grid)  # grid broadcasts against y[..., None]
    is_best = dist == dist.min(axis=-1, keepdims=True)
    first = np.argmax(is_best, axis=-1)
    nxt = np.minimum(first + 1, dist.shape[-1] - 1)
    next_also = np.take_along_axis(is_best, nxt[..., None], axis=-1)[..., 0] & (nxt != first)
    k = first + (next_also & (first % 2 == 1))
    top = np.broadcast_to(grid, dist.shape)[..., -1]
    return np.where(y >= top, dist.shape[-1] - 1, k)


def _row_chunked(fn):
    """Apply a row-wise quantizer to slices of rows to bound the float64 temporaries."""

    def wrapper(x):
        x = np.asarray(x)
        step = max(1, (1 << 21) // max(1, x.shape[1] if x.ndim == 2 else 1))
        if x.ndim != 2 or x.shape[0] <= step:
            return fn(x)
        parts = [fn(x[r:r + step]) for r in range(0, x.shape[0], step)]
        return tuple(np.concatenate(p, axis=0) for p in zip(*parts))

    wrapper.__name__ = fn.__name__
    wrapper.__doc__ = fn.__doc__
    return wrapper


def _blocks(x: np.ndarray, b: int) -> np.ndarray:
    x = np.asarray(x)
    if x.ndim != 2 or x.shape[1] % b != 0:
        raise ValueError(f"expected a 2-D array whose last axis is a multiple of {b}")
    return x.astype(np.float64).reshape(x.shape[0], x.shape[1] // b, b)


# ----------------------------------------------------------------------------------------
# MXFP4
# ----------------------------------------------------------------------------------------
@_row_chunked
def mxfp4_quantize(x: np.ndarray):
    """MXFP4-quantize ``x`` (rows x K, K % 32 == 0) along its last axis.

    Returns ``(codes, scales)``: codes uint8 rows x K (one nibble each), scales uint8
    rows x K/32 holding the E8M0 code (exponent + 127).
    """
    xb = _blocks(x, MX_BLOCK)
    a = np.abs(xb)
    amax = a.max(axis=-1)
    _, ex = np.frexp(amax)  # amax = f * 2**ex with f in [0.5, 1) -> floor(log2 amax) = ex - 1
    e = np.where(amax > 0, ex - 1 - 2, -E8M0_BIAS)
    e = np.clip(e, -E8M0_BIAS, E8M0_BIAS)
    y = np.ldexp(a, -e[..., None])  # exact: a power-of-two rescale in float64
    k = _nearest_ties_even(y, E2M1_MAGNITUDES)
    sign = np.signbit(xb).astype(np.uint8)
    codes = (sign << 3) | k.astype(np.uint8)
    return codes.reshape(x.shape[0], -1), (e + E8M0_BIAS).astype(np.uint8)


def mxfp4_dequantize(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """float64 values of MXFP4 codes (rows x K) and E8M0 scales (rows x K/32)."""
    codes = np.asarray(codes)
    mag = E2M1_MAGNITUDES[codes & 7]
    val = np.where(codes & 8, -mag, mag).reshape(codes.shape[0], -1, MX_BLOCK)
    e = scales.astype(np.int64) - E8M0_BIAS
    return np.ldexp(val, e[..., None]).reshape(codes.shape)


# ----------------------------------------------------------------------------------------
# HiF4
# ----------------------------------------------------------------------------------------
@_row_chunked
def hif4_quantize(x: np.ndarray):
    """HiF4-quantize ``x`` (rows x K, K % 64 == 0) along its last axis (readings H1-H6).

    Returns ``(codes, meta)``: codes uint8 rows x K (sign << 3 | k), meta uint32 rows x K/64.
    """
    xb = _blocks(x, HIF4_BLOCK)
    rows, nb, _ = xb.shape
    a = np.abs(xb)
    # level 1: smallest E6M2 value s1 with 1.75 * s1 >= max|x|
    v = e6m2_values()
    c1 = np.searchsorted(1.75 * v, a.max(axis=-1), side="left")
    c1 = np.minimum(c1, 255)
    s1 = v[c1]  # rows x nb
    # level 2: groups of 8
    a8 = a.reshape(rows, nb, 8, 8).max(axis=-1)
    b2 = a8 <= 1.75 * s1[..., None] / 2.0  # rows x nb x 8
    s2 = s1[..., None] * np.where(b2, 0.5, 1.0)
    # level 3: groups of 4 (two per level-2 group)
    a4 = a.reshape(rows, nb, 8, 2, 4).max(axis=-1)
    b3 = a4 <= 1.75 * s2[..., None] / 2.0  # rows x nb x 8 x 2
    s = s2[..., None] * np.where(b3, 0.5, 1.0)
    # elements: nearest k * s / 4, ties to even k
    grid = S1P2_MAGNITUDES * s[..., None, None]  # rows x nb x 8 x 2 x 1 x 8
    k = _nearest_ties_even(a.reshape(rows, nb, 8, 2, 4), grid)
    sign = np.signbit(xb).astype(np.uint8)
    codes = (sign << 3) | k.reshape(rows, nb, 64).astype(np.uint8)
    meta = c1.astype(np.uint64)
    for g in range(8):
        meta |= b2[:, :, g].astype(np.uint64) << np.uint64(8 + g)
    b3f = b3.reshape(rows, nb, 16)
    for h in range(16):
        meta |= b3f[:, :, h].astype(np.uint64) << np.uint64(16 + h)
    return codes.reshape(x.shape[0], -1), meta.astype(np.uint32)


def hif4_meta_fields(meta: np.ndarray):
    """Split HiF4 metadata into (E6M2 code, level-2 bits [..., 8], level-3 bits [..., 16])."""
    meta = np.asarray(meta, dtype=np.uint32)
    c1 = (meta & 0xFF).astype(np.int64)
    b2 = (meta[..., None] >> (8 + np.arange(8, dtype=np.uint32))) & 1
    b3 = (meta[..., None] >> (16 + np.arange(16, dtype=np.uint32))) & 1
    return c1, b2.astype(np.int64), b3.astype(np.int64)


def hif4_dequantize(codes: np.ndarray, meta: np.ndarray) -> np.ndarray:
    """float64 values of HiF4 codes (rows x K) and metadata (rows x K/64)."""
    codes = np.asarray(codes)
    rows = codes.shape[0]
    c1, b2, b3 = hif4_meta_fields(meta)
    s1 = e6m2_values()[c1]  # rows x nb
    shift = b2[..., :, None] + b3.reshape(b3.shape[:-1] + (8, 2))  # rows x nb x 8 x 2
    s = np.ldexp(s1[..., None, None], -shift)
    k = (codes & 7).astype(np.float64).reshape(rows, -1, 8, 2, 4)
    val = k / 4.0 * s[..., None]
    val = np.where((codes & 8).reshape(val.shape) != 0, -val, val)
    return val.reshape(codes.shape)


# ----------------------------------------------------------------------------------------
# format dispatch
# ----------------------------------------------------------------------------------------
FORMATS = ("mxfp4", "hif4")


def block_size(fmt: str) -> int:
    return {"mxfp4": MX_BLOCK, "hif4": HIF4_BLOCK}[fmt]


def quantize(fmt: str, x: np.ndarray):
    """Q along the last axis: ``(codes, scales_or_meta)``."""
    if fmt == "mxfp4":
        return mxfp4_quantize(x)
    if fmt == "hif4":
        return hif4_quantize(x)
    raise ValueError(fmt)


def dequantize(fmt: str, codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    if fmt == "mxfp4":
        return mxfp4_dequantize(codes, scales)
    if fmt == "hif4":
        return hif4_dequantize(codes, scales)
    raise ValueError(fmt)


def pack_nibbles(codes: np.ndarray) -> np.ndarray:
    """Two codes per byte along the last axis, element 2i in the low nibble."""
    codes = np.asarray(codes, dtype=np.uint8)
    return (codes[..., 0::2] | (codes[..., 1::2] << 4)).astype(np.uint8)


def unpack_nibbles(packed: np.ndarray) -> np.ndarray:
    packed = np.asarray(packed, dtype=np.uint8)
    out = np.empty(packed.shape[:-1] + (packed.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = packed & 15
    out[..., 1::2] = packed >> 4
    return out
