"""Rollout-ResQ linear layer (oracle; test infrastructure only).

Follows paper Sec. 3 (Eq. 1), Sec. 4.3 (Eq. 2, Eq. 3, Eq. 4 and the sparsity functions S),
the FP4 training policy of Sec. 1 / Sec. 4.1 (forward and backward at 4 bits) and the cost
model of Sec. 5.4.  Notation: X is m x d (tokens x input features), W is n x d, Y = X W^T.

Readings of points the paper leaves open (also listed in the design notes):

  R1  the residual Delta X = X - Q(X) is formed in float32 (exact for bf16 inputs whose
      quantized value is within range).
  R2  S acts on the quantized residual Q(Delta X) and the residual GEMM multiplies by Q(W)
      (Eq. 4), not by W.
  S1  S_50% is the paper's structured channel-wise sparsity; an element-wise (unstructured)
      50% variant is provided as well.
  S2  a channel is a column of the m x d activation (an input feature); its L2 norm runs over
      all m rows of the call (the residual is taken at tensor level, Sec. 4.3).
  S3  a 32 x 64 block covers 32 rows (tokens) by 64 columns (features); a last row-block with
      fewer than 32 rows is a smaller block.
  S4  ranking uses the sum of squares (same order as the L2 norm); ties go to the lowest
      index; floor(count / 2) items are kept.
  S6  other levels and patterns (Sec. 4.3 defines S_alpha%, S_{M:N} and S^{MxN}_alpha% for
      any alpha, M, N; Sec. 6 leaves levels other than 50% open): alpha is the kept percent,
      floor(count * alpha / 100) items are kept, with the ranking and ties of S4; "k:g" keeps
      the k largest of every g consecutive elements along d (ties to the lower index).
  S5  sums of squares are float64 in a fixed order (stated at each function), so near-ties
      are decided the same way on every implementation that keeps that order.
  T1  backward: dY, W and X are quantized along the contraction axis of each backward GEMM
      (dX = Q_n(dY) Q_n(W), dW = Q_m(dY)^T Q_m(X)), no residual (ResQ is rollout-only).
  Y1  Y, dX and dW are float32: the exact float64 result rounded once.
  Y2  the optional bf16 output is that float32 result rounded again, to the nearest bf16
      (ties to even): the rounding of the float32 result, not of the float64 one.
  W1  the mixed-precision rollout linears of Table 1 keep one operand in its 16-bit form:
      W4A16 is X Q(W)^T and W16A4 is Q(X) W^T, with Q along d as in Eq. 1 (the W4A8 row
      needs an 8-bit activation format that the paper does not name, and is not built).
  F1  the fused producer of the down projection's input (the SwiGLU of the gate and up
      projections, X = silu(G) * U, silu(g) = g / (1 + exp(-g))): X is the bf16 nearest to the
      float64 value of silu(g) * u (ties to even), rounded once, so it is the bf16 activation
      the unfused model would hand to the linear up to that single rounding.
  N1  the fused producer of the qkv and gate/up projections' input, the RMSNorm of the
      residual stream H (bf16, m x d) with gain gamma (bf16, d) and epsilon eps (a float32
      >= 2^-126), as the Qwen2.5 models of Sec. 5.1 apply it before those linears (the paper
      does not spell it out).  Every step is one IEEE float32 operation, rounded to nearest
      even, except the sum of squares, which is exact and then rounded once:
          s = f32(sum_j H_j^2),  mu = f32(s / d),  t = f32(mu + eps),
          q = f32(sqrt(t)),      r = f32(1 / q),
          X_j = bf16(f32(f32(H_j * r) * gamma_j)),
      so X does not depend on any summation order.
"""
from __future__ import annotations

import numpy as np

from . import formats as F

SPARSITY = ("none", "identity", "2:4", "channel50", "block32x64_50", "unstructured50")


def parse_sparsity(kind: str):
    """Family and parameters of a sparsity name (reading S6).

    "none", "identity"; "k:g" (local k of g); "channel<p>", "block32x64_<p>",
    "unstructured<p>" (global, p percent kept)."""
    if kind in ("none", "identity"):
        return kind, None
    if ":" in kind:
        k, g = (int(v) for v in kind.split(":"))
        if g not in (4, 8) or not 1 <= k < g:
            raise ValueError(kind)
        return "local", (k, g)
    for fam, prefix in (("channel", "channel"), ("block", "block32x64_"), ("unstructured", "unstructured")):
        if kind.startswith(prefix) and kind[len(prefix):].isdigit():
            p = int(kind[len(prefix):])
            if not 1 <= p <= 99:
                raise ValueError(kind)
            return fam, p
    raise ValueError(kind)


def kept_fraction(kind: str) -> float:
    """Nominal fraction of Q(Delta X) a sparsity function keeps (1 for identity, 0 for none)."""
    fam, par = parse_sparsity(kind)
    if fam == "none":
        return 0.0
    if fam == "identity":
        return 1.0
    if fam == "local":
        return par[0] / par[1]
    return par / 100.0


# ----------------------------------------------------------------------------------------
# Eq. 2: the activation residual
# ----------------------------------------------------------------------------------------
def residual(x: np.ndarray, xhat: np.ndarray) -> np.ndarray:
    """Delta X = X - Q(X) in float32 (Eq. 2, reading R1)."""
    return np.asarray(x, np.float32) - np.asarray(xhat).astype(np.float32)


# ----------------------------------------------------------------------------------------
# Sec. 4.3: sparsity functions applied to Q(Delta X)
# ----------------------------------------------------------------------------------------
def keep_k_of_g(rhat: np.ndarray, k: int, g: int) -> np.ndarray:
    """S_{k:g}: in every group of g consecutive elements along d, keep the k largest |value|.

    An element's rank in its group is the number of elements that beat it: larger magnitude,
    or equal magnitude and a lower index.  Ranks 0 .. k-1 are kept.
    """
    m, d = rhat.shape
    a = np.abs(rhat).reshape(m, d // g, g)
    rank = np.zeros(a.shape, dtype=np.int64)
    for i in range(g):
        for j in range(g):
            if j == i:
                continue
            beats = (a[..., j] > a[..., i]) | ((a[..., j] == a[..., i]) & (j < i))
            rank[..., i] += beats
    return (rank < k).reshape(m, d)


def keep_2_4(rhat: np.ndarray) -> np.ndarray:
    """S_{2:4}: in every group of 4 consecutive elements along d, keep the 2 largest |value|."""
    return keep_k_of_g(rhat, 2, 4)


def channel_keys(rhat: np.ndarray) -> np.ndarray:
    """Sum of squares of every column, accumulated in float64 over rows i = 0, 1, ..., m-1."""
    acc = np.zeros(rhat.shape[1], dtype=np.float64)
    for i in range(rhat.shape[0]):
        acc = acc + rhat[i].astype(np.float64) ** 2
    return acc


def _top(keys: np.ndarray, pct: int = 50) -> np.ndarray:
    """Boolean mask of the floor(len * pct / 100) largest keys; ties go to the lower index."""
    idx = np.arange(keys.size)
    order = np.lexsort((idx, -keys))  # primary: key descending, secondary: index ascending
    keep = np.zeros(keys.size, dtype=bool)
    keep[order[: keys.size * pct // 100]] = True
    return keep


def keep_channel(rhat: np.ndarray, pct: int = 50):
    """S_alpha% (structured, channel-wise): keep the top alpha% of the d channels by L2 norm."""
    ch = _top(channel_keys(rhat), pct)
    return np.broadcast_to(ch[None, :], rhat.shape).copy(), ch


def keep_channel50(rhat: np.ndarray):
    """S_50%: keep the top half of the d channels by L2 norm."""
    return keep_channel(rhat, 50)


def block_keys(rhat: np.ndarray, fmt: str) -> np.ndarray:
    """Sum of squares of every 32 x 64 block, shape (ceil(m/32), d/64).

    Order (reading S5): rows of the block in increasing order; within a row, the block's
    format scale blocks in increasing column order (one for HiF4, two 32-wide halves for
    MXFP4), each added as its own sum.  Every inner sum is exact in float64, in any order:
    - MXFP4: each square is q^2 2^(2E) with q in the E2M1 grid, i.e. an integer multiple of
      2^(2E-2) below 2^8, so 32 of them add to an integer multiple of 2^(2E-2) below 2^13;
    - HiF4: each value is k (4+m) 2^(e-35-b) with k <= 7, m <= 3 and the element's own
      level-2/3 shift b in 0..2 (b differs inside a block), so each square is an integer
      multiple of 2^(2e-74) below 2401 * 2^4, and 64 of them add to an integer below 2^22 in
      those units.
    So the grouping by scale block is the plain sequential sum of the block's squares with
    its exact partial sums formed first; it can differ from an element-by-element sequential
    order only where a row-level addition rounds, and it is the grouping the GPU forms from
    its per-scale-block partials.
    """
    m, d = rhat.shape
    sb = F.block_size(fmt)
    sq = rhat.astype(np.float64) ** 2
    inner = sq.reshape(m, d // sb, sb).sum(axis=-1)  # exact per scale block
    per64 = inner.reshape(m, d // 64, 64 // sb)
    nI = (m + 31) // 32
    keys = np.zeros((nI, d // 64), dtype=np.float64)
    for bi in range(nI):
        acc = np.zeros(d // 64, dtype=np.float64)
        for i in range(32 * bi, min(m, 32 * bi + 32)):
            for q in range(64 // sb):
                acc = acc + per64[i, :, q]
        keys[bi] = acc
    return keys


def keep_block(rhat: np.ndarray, fmt: str, pct: int = 50):
    """S^{32x64}_alpha%: keep the top alpha% of the 32 x 64 blocks by L2 norm (row-major index)."""
    keys = block_keys(rhat, fmt)
    blk = _top(keys.ravel(), pct).reshape(keys.shape)
    elem = np.repeat(np.repeat(blk, 32, axis=0)[: rhat.shape[0]], 64, axis=1)
    return elem, blk


def keep_block50(rhat: np.ndarray, fmt: str):
    """S^{32x64}_50%: keep the top half of the 32 x 64 blocks by L2 norm."""
    return keep_block(rhat, fmt, 50)


def keep_unstructured(rhat: np.ndarray, pct: int = 50) -> np.ndarray:
    """Element-wise alpha%: keep the floor(m*d*alpha/100) largest |value| (row-major index)."""
    return _top(np.abs(rhat).ravel(), pct).reshape(rhat.shape)


def keep_unstructured50(rhat: np.ndarray) -> np.ndarray:
    """Element-wise 50%: keep the floor(m*d/2) largest |value| of the tensor."""
    return keep_unstructured(rhat, 50)


def sparsify(kind: str, fmt: str, rcodes: np.ndarray, rhat: np.ndarray):
    """Apply S to Q(Delta X).

    Returns ``(codes, keep, groups)``: the residual codes with pruned elements set to the +0
    code, the element keep mask, and the kept channels (d,) or blocks (ceil(m/32), d/64) for
    the channel and block kinds (None otherwise).
    """
    groups = None
    fam, par = parse_sparsity(kind)
    if fam == "identity":
        keep = np.ones(rhat.shape, dtype=bool)
    elif fam == "local":
        keep = keep_k_of_g(rhat, *par)
    elif fam == "channel":
        keep, groups = keep_channel(rhat, par)
    elif fam == "block":
        keep, groups = keep_block(rhat, fmt, par)
    elif fam == "unstructured":
        keep = keep_unstructured(rhat, par)
    else:
        raise ValueError(kind)
    return np.where(keep, rcodes, 0).astype(np.uint8), keep, groups


def pack_bits(mask: np.ndarray) -> np.ndarray:
    """Bit b of byte i along the last axis is element 8i + b."""
    return np.packbits(np.asarray(mask, dtype=bool), axis=-1, bitorder="little")


# ----------------------------------------------------------------------------------------
# forward: Eq. 1 (S = none), Eq. 3 (S = identity), Eq. 4 (S = one of the sparsifiers)
# ----------------------------------------------------------------------------------------
def resq_quantize_residual(fmt: str, sparsity: str, x: np.ndarray) -> dict:
    """Q(X), Delta X, Q(Delta X) and S(Q(Delta X)) for activations x (m x d, float32)."""
    qx_codes, qx_scales = F.quantize(fmt, x)
    xhat = F.dequantize(fmt, qx_codes, qx_scales)
    out = {"qx_codes": qx_codes, "qx_scales": qx_scales, "xhat": xhat}
    if sparsity == "none":
        return out
    r = residual(x, xhat)
    qr_codes, qr_scales = F.quantize(fmt, r)
    rhat = F.dequantize(fmt, qr_codes, qr_scales)
    sr_codes, keep, groups = sparsify(sparsity, fmt, qr_codes, rhat)
    out.update(r=r, qr_codes_dense=qr_codes, qr_scales=qr_scales, qr_codes=sr_codes,
               keep=keep, groups=groups, srhat=np.where(keep, rhat, 0.0))
    return out


def resq_forward(fmt: str, sparsity: str, x: np.ndarray, w: np.ndarray) -> dict:
    """Y = Q(X) Q(W)^T + S(Q(Delta X)) Q(W)^T, float64 products rounded to float32 once."""
    out = resq_quantize_residual(fmt, sparsity, x)
    qw_codes, qw_scales = F.quantize(fmt, w)
    what = F.dequantize(fmt, qw_codes, qw_scales)
    y = out["xhat"] @ what.T
    if sparsity != "none":
        y = y + out["srhat"] @ what.T
    out.update(qw_codes=qw_codes, qw_scales=qw_scales, what=what, y=y.astype(np.float32),
               y64=y)
    return out


def w4a16_forward(fmt: str, x: np.ndarray, w: np.ndarray) -> dict:
    """Weight-only FP4 rollout linear (Table 1, "W4A16"): the weights are quantized, the
    activations stay in their 16-bit form.  Y = X Q(W)^T with Q(W) blocked along d, float64
    products rounded to float32 once."""
    what = F.dequantize(fmt, *F.quantize(fmt, w))
    y = np.asarray(x, np.float64) @ what.astype(np.float64).T
    return {"what": what, "y64": y, "y": y.astype(np.float32)}


def w16a4_forward(fmt: str, x: np.ndarray, w: np.ndarray) -> dict:
    """Activation-only FP4 rollout linear (Table 1, "W16A4"): the activations are quantized
    (blocked along d, as in Eq. 1), the weights stay in their 16-bit form.  Y = Q(X) W^T,
    float64 products rounded to float32 once."""
    xhat = F.dequantize(fmt, *F.quantize(fmt, x))
    y = xhat.astype(np.float64) @ np.asarray(w, np.float64).T
    return {"xhat": xhat, "y64": y, "y": y.astype(np.float32)}


def round_to_bf16(y32: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of finite float32 values, round to nearest, ties to even (reading Y2).

    A bf16 keeps the sign, the 8 exponent bits and the top 7 fraction bits of a float32; the
    16 dropped bits are compared with half of the kept part's last place."""
    u = np.asarray(y32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    kept, dropped = u >> 16, u & 0xFFFF
    up = (dropped > 0x8000) | ((dropped == 0x8000) & ((kept & 1) == 1))
    return (kept + up).astype(np.uint16)


def round_f64_to_bf16(v: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of finite float64 values, nearest, ties to even, in one rounding.

    The bf16 grid spacing at |v| in [2^e, 2^(e+1)) is 2^(e-7) (e >= -126; below that the
    subnormal spacing 2^-133): v / spacing is exact in float64, rounded half to even with
    rint, and scaled back.  Magnitudes that round past the largest finite bf16 become inf."""
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    # log2 may land one off near powers of two: fix e so that 2^e <= a < 2^(e+1)
    e = np.where(np.exp2(e) > a, e - 1, e)
    e = np.where(np.exp2(e + 1) <= a, e + 1, e)
    step = np.exp2(np.maximum(e, -126.0) - 7.0)
    q = np.rint(a / step) * step
    f32 = np.where(q > float(np.finfo(np.float32).max), np.inf, q).astype(np.float32)
    bits = (f32.view(np.uint32) >> 16).astype(np.uint16)
    return bits | np.where(np.signbit(v), np.uint16(0x8000), np.uint16(0))


def swiglu_bf16(g: np.ndarray, u: np.ndarray) -> np.ndarray:
    """X = silu(G) * U as bf16 bit patterns (reading F1): float64 value, rounded once."""
    g = np.asarray(g, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    return round_f64_to_bf16(g / (1.0 + np.exp(-g)) * u)


def _round_dyadic_to_f32(num: int, exp: int) -> np.float32:
    """The float32 nearest to num * 2^exp (num >= 0 an integer), ties to even, with float32's
    subnormals (spacing 2^-149) and overflow to inf."""
    if num == 0:
        return np.float32(0.0)
    msb = num.bit_length() - 1 + exp            # 2^msb <= value < 2^(msb + 1)
    unit = max(msb - 23, -149)                  # spacing of the float32 grid at the value
    q = num
    if unit > exp:                              # drop the bits below the grid, nearest even
        drop = unit - exp
        q, rem = divmod(num, 1 << drop)
        half = 1 << (drop - 1)
        if rem > half or (rem == half and q & 1):
            q += 1
    else:
        unit = exp                              # on the grid already: num < 2^24
    if q * 2.0**unit >= 2.0**128:
        return np.float32(np.inf)
    return np.float32(np.ldexp(float(q), unit))  # q <= 2^24: exact


def exact_square_sums_f32(h: np.ndarray) -> np.ndarray:
    """Per row of h (float32 values on the bf16 grid), the float32 nearest to the exact sum of
    the squares (reading N1).  A bf16 value is an integer of at most 8 bits times a power of
    two, so each square is an integer of at most 16 bits times 2^(2e); the squares of one
    exponent are added as integers, the exponents' sums are combined exactly as one Python
    integer, and that is rounded once."""
    h = np.asarray(h, dtype=np.float32)
    assert (h.view(np.uint32) & 0xFFFF == 0).all(), "H must be bf16 values"
    frac, ex = np.frexp(h.astype(np.float64))   # h = frac * 2^ex, |frac| in [0.5, 1)
    mant = np.abs(np.rint(frac * 256.0)).astype(np.int64)  # h = +-mant * 2^(ex - 8), exactly
    e2 = 2 * (ex.astype(np.int64) - 8)          # h^2 = mant^2 * 2^e2
    out = np.zeros(h.shape[0], dtype=np.float32)
    for i in range(h.shape[0]):
        nz = mant[i] != 0
        if not nz.any():
            continue
        lo = int(e2[i][nz].min())
        per_exp = np.zeros(int(e2[i][nz].max()) - lo + 1, dtype=np.int64)
        np.add.at(per_exp, e2[i][nz] - lo, mant[i][nz] ** 2)   # < 2^16 each: exact in int64
        total = sum(int(v) << k for k, v in enumerate(per_exp.tolist()) if v)
        out[i] = _round_dyadic_to_f32(total, lo)
    return out


def rmsnorm_bf16(h: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """X = RMSNorm(H) * gamma as bf16 bit patterns (reading N1).  h: m x d float32 values on
    the bf16 grid, gamma: d values on the bf16 grid, eps: a float32 >= 2^-126."""
    h = np.asarray(h, dtype=np.float32)
    gamma = np.asarray(gamma, dtype=np.float32)
    d = h.shape[1]
    assert d <= 2**24 and np.float32(eps) >= np.float32(2.0**-126)
    s = exact_square_sums_f32(h)
    mu = s / np.float32(d)
    t = mu + np.float32(eps)
    q = np.sqrt(t)
    r = np.float32(1.0) / q
    y = h * r[:, None]
    x = y * gamma[None, :]
    return round_to_bf16(x)


# ----------------------------------------------------------------------------------------
# FP4 training-policy backward (reading T1)
# ----------------------------------------------------------------------------------------
def resq_backward(fmt: str, dy: np.ndarray, x: np.ndarray, w: np.ndarray) -> dict:
    """dX = Q_n(dY) Q_n(W) and dW = Q_m(dY)^T Q_m(X), each quantized along its contraction.

    dy is m x n, x is m x d, w is n x d.  Q_a(T) means T quantized in blocks along axis a.
    """
    dyn = F.dequantize(fmt, *F.quantize(fmt, dy))            # blocks along n
    wn_t = F.dequantize(fmt, *F.quantize(fmt, w.T))          # d x n, blocks along n
    dym_t = F.dequantize(fmt, *F.quantize(fmt, dy.T))        # n x m, blocks along m
    xm_t = F.dequantize(fmt, *F.quantize(fmt, x.T))          # d x m, blocks along m
    dx = dyn @ wn_t.T
    dw = dym_t @ xm_t.T
    return {"dx": dx.astype(np.float32), "dw": dw.astype(np.float32), "dx64": dx, "dw64": dw}


# ----------------------------------------------------------------------------------------
# Sec. 5.4: overhead cost model (FLOPs)
# ----------------------------------------------------------------------------------------
def flops_dense(m: int, d: int, n: int) -> int:
    """A dense GEMM Y = X W^T costs 2mdn FLOPs."""
    return 2 * m * d * n


def flops_resq(m: int, d: int, n: int, sparsity: str) -> int:
    """Algorithmic FLOPs of a ResQ linear: the FP4 main GEMM plus the kept residual part.

    S_2:4, S_50% (channel or element-wise) and the 50% block pattern keep half of the residual
    (mdn); the identity keeps all of it (2mdn); no residual adds nothing.  Other levels and
    patterns cost their nominal kept fraction of 2mdn (reading S6).
    """
    main = flops_dense(m, d, n)
    extra = round(2 * m * d * n * kept_fraction(sparsity))
    return main + extra


def effective_cost(m: int, d: int, n: int, sparsity: str, fp4_speedup: float = 4.0) -> float:
    """Sec. 5.4 cost in FP16-equivalent FLOPs, FP4 GEMMs taken as fp4_speedup times cheaper."""
    return flops_resq(m, d, n, sparsity) / fp4_speedup


def speedup_vs_fp16(sparsity: str, fp4_speedup: float = 4.0) -> float:
    m = d = n = 1
    return flops_dense(m, d, n) / effective_cost(m, d, n, sparsity, fp4_speedup)
