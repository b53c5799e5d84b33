"""GPU <-> oracle parity through the C ABI: bit-exact codes, scales and masks; float32
outputs within a normwise relative error of 1e-5.  Shapes span several tiles and ragged
tails; inputs are seeded synthetic data with outlier channels plus adversarial blocks."""
import numpy as np
import pytest

from oracle import formats as F
from oracle import resq as Q
from synth import activations, bf16_bits_to_f32, f32_to_bf16_bits, grad_output, rng_tree, weights
from _gpu_util import (assert_close, assert_codes_equal, assert_scales_equal, dev_bf16, dev_f32,
                       host, log, pack_bits)

pytestmark = pytest.mark.gpu

FMTS = ["mxfp4", "hif4"]


def _adversarial_bits(rows, cols, seed):
    """bf16 rows: outlier data plus zero rows, -0, subnormals, ties, a single outlier, a large
    in-range block and exact E2M1/S1P2 midpoints."""
    rng = rng_tree(seed, 1)[0]
    x = bf16_bits_to_f32(activations(rng, rows, cols, 0.02, 50.0)).copy()
    if rows >= 8:
        x[0] = 0.0
        x[1] = -0.0
        x[2, :] = bf16_bits_to_f32(np.arange(1, cols + 1, dtype=np.uint16) % 128)  # subnormals
        x[3, :] = 1.0  # all ties
        x[4, :] = 0.01
        x[4, cols // 2] = 300.0  # single outlier
        x[5, :] = 2.0 ** 20 * np.sign(x[5])  # large, in range
        x[6, :] = np.resize(np.array([6.0, 5.0, 3.5, 2.5, 1.75, 1.25, 0.75, 0.25], np.float32), cols)  # MX midpoints
        x[7, :] = np.resize(np.array([1.75, 1.625, 1.375, 1.125, 0.875, 0.625, 0.375, 0.125], np.float32), cols)
    return f32_to_bf16_bits(x)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("rows,cols", [(1, 64), (37, 256), (300, 2048), (8, 11008)])
def test_quantize_rows_bf16(fmt, rows, cols):
    import paper_2607_26515_amd as P
    log(f"quantize rows bf16 {fmt} {rows}x{cols}")
    bits = _adversarial_bits(rows, cols, seed=rows + cols)
    codes, scales = P.quantize(dev_bf16(bits), fmt, axis=1)
    oc, os_ = F.quantize(fmt, bf16_bits_to_f32(bits))
    assert_codes_equal(codes, oc, "codes")
    assert_scales_equal(fmt, scales, os_, "scales")


@pytest.mark.parametrize("fmt", FMTS)
def test_quantize_rows_f32_midpoints(fmt):
    import paper_2607_26515_amd as P
    log(f"quantize rows f32 {fmt}")
    rng = np.random.default_rng(21)
    x = (rng.standard_normal((64, 512)) * np.exp2(rng.integers(-30, 30, (64, 1)))).astype(np.float32)
    x[:8] = np.float32(1.0)
    x[:8, 1:9] = np.float32(0.375)
    x[8:16] = (rng.integers(-28, 29, (8, 512)) / 16.0).astype(np.float32)  # many exact ties
    codes, scales = P.quantize(dev_f32(x), fmt, axis=1)
    oc, os_ = F.quantize(fmt, x)
    assert_codes_equal(codes, oc, "codes")
    assert_scales_equal(fmt, scales, os_, "scales")


def test_quantize_mx_block_edges():
    """MXFP4 blocks built around fixed shared exponents E (the block holds 4 * 2^E, so E is
    floor(log2 amax) - 2): every E2M1 tie and threshold, values that saturate at 6, +-0 and
    near-tie neighbours, at E from -127 (2^E subnormal) to 124.  Codes and scales must match
    the oracle exactly."""
    import paper_2607_26515_amd as P
    log("quantize mx block edges")
    ladder = np.array([4.0, -4.0, 7.99, -7.0, 6.0, 6.5, 5.0, 3.5, 2.5, 1.75, 1.25, 0.75, 0.25, -0.25,
                       0.2499, 0.2501, 0.0, -0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 5.0001, 4.9999, 0.74999,
                       0.75001, -1.25, -2.5, -3.5, -5.0, 0.125], dtype=np.float64)
    assert ladder.size == 32
    exps = [-127, -126, -125, -100, -20, -1, 0, 1, 7, 60, 120, 124]
    rng = np.random.default_rng(5)
    rows = []
    for e in exps:
        for r in range(4):
            perm = ladder if r == 0 else rng.permutation(ladder)
            rows.append(np.concatenate([perm, -perm]) * 2.0 ** e)  # two blocks per row
    x = np.array(rows, dtype=np.float32)
    codes, scales = P.quantize(dev_f32(x), "mxfp4", axis=1)
    oc, os_ = F.quantize("mxfp4", x)
    assert_codes_equal(codes, oc, "codes")
    assert_scales_equal("mxfp4", scales, os_, "scales")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("rows,cols", [(64, 1), (128, 37), (192, 100), (2048, 130)])
def test_quantize_cols(fmt, rows, cols):
    import paper_2607_26515_amd as P
    if rows % F.block_size(fmt):
        pytest.skip("rows must be a multiple of the block size")
    log(f"quantize cols {fmt} {rows}x{cols}")
    bits = _adversarial_bits(rows, cols, seed=3 * rows + cols)
    codes, scales = P.quantize(dev_bf16(bits), fmt, axis=0)
    oc, os_ = F.quantize(fmt, bf16_bits_to_f32(bits).T.copy())
    assert_codes_equal(codes, oc, "codes")
    assert_scales_equal(fmt, scales, os_, "scales")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["none", "identity", "2:4"])
@pytest.mark.parametrize("m,d", [(1, 64), (37, 512), (256, 2048)])
def test_residual_sparsify_local(fmt, sp, m, d):
    import paper_2607_26515_amd as P
    log(f"residual_sparsify {fmt} {sp} {m}x{d}")
    bits = _adversarial_bits(m, d, seed=m * 7 + d)
    out = P.residual_sparsify(dev_bf16(bits), fmt, sp)
    o = Q.resq_quantize_residual(fmt, sp, bf16_bits_to_f32(bits))
    assert_codes_equal(out["qx_codes"], o["qx_codes"], "Q(X) codes")
    assert_scales_equal(fmt, out["qx_scales"], o["qx_scales"], "Q(X) scales")
    if sp != "none":
        assert_codes_equal(out["qr_codes"], o["qr_codes"], "S(Q(dX)) codes")
        assert_scales_equal(fmt, out["qr_scales"], o["qr_scales"], "Q(dX) scales")
        assert np.array_equal(host(out["keep_mask"]), pack_bits(o["keep"]))


def _linear_case(fmt, sp, m, d, n, seed):
    import paper_2607_26515_amd as P
    rx, rw = rng_tree(seed, 2)
    xb = activations(rx, m, d, 0.01, 50.0)
    wb = weights(rw, n, d)
    qw_codes, qw_scales = P.quantize(dev_bf16(wb), fmt, axis=1)
    y = P.linear_fwd(dev_bf16(xb), qw_codes, qw_scales, fmt, sp)
    o = Q.resq_forward(fmt, sp, bf16_bits_to_f32(xb), bf16_bits_to_f32(wb))
    return host(y), o


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["none", "identity", "2:4"])
@pytest.mark.parametrize("m,d,n", [(1, 64, 1), (16, 256, 100), (37, 512, 33), (100, 2048, 300),
                                   (256, 1024, 640)])
def test_linear_fwd(fmt, sp, m, d, n):
    log(f"linear_fwd {fmt} {sp} m={m} d={d} n={n}")
    y, o = _linear_case(fmt, sp, m, d, n, seed=m + d + n)
    assert y.shape == (m, n)
    assert_close(y, o["y64"], f"Y {fmt} {sp}")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["none", "2:4"])
@pytest.mark.parametrize("m,d,n", [(16, 2048, 2048), (256, 2048, 2560), (256, 11008, 2048), (37, 512, 100)])
def test_linear_fwd_prepared_matches_unprepared(fmt, sp, m, d, n):
    """Prepared weights give bit-identical Y to the K-major Q(W) path, and match the oracle."""
    import paper_2607_26515_amd as P
    log(f"linear_fwd_prepared {fmt} {sp} m={m} d={d} n={n}")
    rx, rw = rng_tree(m * 3 + n, 2)
    xb, wb = activations(rx, m, d, 0.01, 50.0), weights(rw, n, d)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    x = dev_bf16(xb)
    y1 = host(P.linear_fwd(x, qc, qs, fmt, sp))
    wprep = P.prepare_weights(qc, qs, fmt)
    y2 = host(P.linear_fwd_prepared(x, wprep, n, fmt, sp))
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))
    if m * d * n <= 2**31:
        o = Q.resq_forward(fmt, sp, bf16_bits_to_f32(xb), bf16_bits_to_f32(wb))
        assert_close(y2, o["y64"], "Y")


@pytest.mark.parametrize("sp", ["none", "2:4"])
@pytest.mark.parametrize("d", [32, 96, 480])
def test_linear_fwd_mxfp4_half_step(sp, d):
    """MXFP4 contraction lengths that end in a half (32-element) MFMA step."""
    log(f"linear_fwd mxfp4 half step {sp} d={d}")
    y, o = _linear_case("mxfp4", sp, 45, d, 77, seed=d)
    assert_close(y, o["y64"], "Y")


@pytest.mark.parametrize("fmt", FMTS)
def test_linear_fwd_is_deterministic(fmt):
    import paper_2607_26515_amd as P
    log(f"determinism {fmt}")
    rx, rw = rng_tree(99, 2)
    xb, wb = activations(rx, 130, 2048, 0.01, 50.0), weights(rw, 700, 2048)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    x = dev_bf16(xb)
    y1 = host(P.linear_fwd(x, qc, qs, fmt, "2:4"))
    y2 = host(P.linear_fwd(x, qc, qs, fmt, "2:4"))
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("m,d,n", [(64, 96, 64), (128, 33, 192), (256, 130, 128), (96, 40, 160)])
def test_linear_bwd(fmt, m, d, n):
    import paper_2607_26515_amd as P
    b = F.block_size(fmt)
    log(f"linear_bwd {fmt} m={m} d={d} n={n}")
    rx, rw, rg = rng_tree(m + n + d, 3)
    xb, wb, gb = activations(rx, m, d, 0.01, 50.0), weights(rw, n, d), grad_output(rg, m, n)
    if m % b or n % b:
        # both GEMMs contract over a blocked axis (n for dX, m for dW): refused before any launch
        with pytest.raises(P.ResqError, match="needs"):
            P.linear_bwd(dev_bf16(gb), dev_bf16(xb), dev_bf16(wb), fmt)
        return
    dx, dw = P.linear_bwd(dev_bf16(gb), dev_bf16(xb), dev_bf16(wb), fmt)
    o = Q.resq_backward(fmt, bf16_bits_to_f32(gb), bf16_bits_to_f32(xb), bf16_bits_to_f32(wb))
    assert_close(host(dx), o["dx64"], "dX")
    assert_close(host(dw), o["dw64"], "dW")


@pytest.mark.parametrize("fmt", FMTS)
def test_linear_bwd_k_groups(fmt):
    """The dW GEMM of m = 8384 (131 K steps), n = d = 128 runs 64 x 64 tiles unsplit with four
    K groups (MXFP4; two for HiF4) and four stages: three K steps in the last stage."""
    import paper_2607_26515_amd as P
    m, d, n = 8384, 128, 128
    log(f"linear_bwd k groups {fmt} m={m} d={d} n={n} dW plan {P.gemm_plan(fmt, n, d, m, False)}")
    rx, rw, rg = rng_tree(m + n + d + 1, 3)
    xb, wb, gb = activations(rx, m, d, 0.01, 50.0), weights(rw, n, d), grad_output(rg, m, n)
    dx, dw = P.linear_bwd(dev_bf16(gb), dev_bf16(xb), dev_bf16(wb), fmt)
    o = Q.resq_backward(fmt, bf16_bits_to_f32(gb), bf16_bits_to_f32(xb), bf16_bits_to_f32(wb))
    assert_close(host(dx), o["dx64"], "dX")
    assert_close(host(dw), o["dw64"], "dW")


@pytest.mark.parametrize("sp", ["none", "2:4"])
@pytest.mark.parametrize("fmt,m,d,n", [
    ("mxfp4", 64, 320, 128),    # 5 K steps, two K groups: the last stage is half empty
    ("mxfp4", 64, 8384, 96),    # 64 x 128 tiles, K split in four (33, 33, 33, 32 steps)
    ("mxfp4", 512, 8384, 1152),  # 64 x 128 tiles, K split in three (44, 44, 43 steps)
    ("mxfp4", 1024, 8384, 1152),  # more workgroups than CUs: four K groups, two stages
    ("hif4", 64, 320, 128),     # 5 K steps, two K groups
    ("hif4", 32, 8384, 64),     # 64 x 128 tiles, K split in four, two K groups each
    ("hif4", 640, 320, 2048),   # more small tiles than CUs, short K: one K group, two stages
    ("hif4", 640, 8384, 2048),  # more small tiles than CUs, long K: two K groups, two stages
    ("mxfp4", 640, 320, 2048),  # more small tiles than CUs, short K: one K group, four stages
    ("mxfp4", 256, 2048, 22016),  # 64 x 128 tiles without a split (MXFP4 decode, wide N)
])
def test_linear_fwd_k_groups(fmt, sp, m, d, n):
    """Decode-sized grids run K groups (several wave groups splitting each stage's K steps)
    or 64 x 128 tiles with a K split; K lengths that leave the last stage partly empty, a
    ragged K split and the two-stage plan must all match the oracle."""
    log(f"linear_fwd k groups {fmt} {sp} m={m} d={d} n={n}")
    y, o = _linear_case(fmt, sp, m, d, n, seed=m + 3 * d + n)
    assert_close(y, o["y64"], f"Y {fmt} {sp}")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["none", "2:4", "unstructured50"])
@pytest.mark.parametrize("m,d,n", [(37, 512, 100), (256, 2048, 2560), (32, 8384, 64),
                                   (1024, 2048, 640)])
def test_linear_fwd_prepared_bf16(fmt, sp, m, d, n):
    """bf16 output: the float32 result rounded to bf16 (nearest, ties to even) by the GEMM's
    epilogue, also on the split-K path (m=32, d=8384)."""
    import torch
    import paper_2607_26515_amd as P
    log(f"linear_fwd_prepared bf16 {fmt} {sp} m={m} d={d} n={n}")
    rx, rw = rng_tree(m * 5 + n + d, 2)
    xb, wb = activations(rx, m, d, 0.01, 50.0), weights(rw, n, d)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    x = dev_bf16(xb)
    wprep = P.prepare_weights(qc, qs, fmt)
    y32 = P.linear_fwd_prepared(x, wprep, n, fmt, sp)
    yb = P.linear_fwd_prepared(x, wprep, n, fmt, sp, out="bf16")
    assert yb.dtype == torch.int16 and yb.shape == (m, n)
    got = host(yb).view(np.uint16)
    # the epilogue's rounding is the bf16 rounding of the float32 result, bit for bit
    want_from_f32 = host(y32.cpu().to(torch.bfloat16).view(torch.int16)).view(np.uint16)
    assert np.array_equal(got, want_from_f32)
    o = Q.resq_forward(fmt, sp, bf16_bits_to_f32(xb), bf16_bits_to_f32(wb))
    assert_close(host(y32), o["y64"], "Y float32")
    # bf16 keeps 8 significant bits: unit roundoff 2^-9, plus the float32 path's error
    assert_close(bf16_bits_to_f32(got), o["y64"], "Y bf16", tol=2.0**-8)
    ob = Q.round_to_bf16(o["y"])
    diff = np.abs(got.astype(np.int32) - ob.astype(np.int32))
    big = np.abs(o["y64"]) > 2.0**-4 * np.sqrt(np.mean(o["y64"] ** 2))
    assert diff[big].max(initial=0) <= 1, "bf16 outputs more than one step from the oracle's"
    assert np.mean(diff == 0) > 0.99


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("m,d,n", [(37, 512, 102), (256, 2048, 2558), (1024, 512, 4102)])
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_linear_fwd_output_layouts(fmt, m, d, n, out):
    """The GEMM stores Y through LDS as row segments, 16 bytes per lane where Y and ldy allow
    it and element by element otherwise.  A strided Y (ldy not a multiple of 4), a Y that
    starts 4 bytes into its buffer and a width that is not a multiple of 4 must give the bits
    of the contiguous result and leave the buffer outside Y untouched.  The shapes run the
    small (K groups), the decode-width and the large-tile plans."""
    import torch
    import paper_2607_26515_amd as P
    log(f"linear_fwd output layouts {fmt} m={m} d={d} n={n} out={out}")
    rx, rw = rng_tree(m + 7 * n + d, 2)
    xb, wb = activations(rx, m, d, 0.01, 50.0), weights(rw, n, d)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    x = dev_bf16(xb)
    wprep = P.prepare_weights(qc, qs, fmt)
    ref = host(P.linear_fwd_prepared(x, wprep, n, fmt, "2:4", out=out))
    dt = torch.float32 if out == "f32" else torch.int16
    sentinel = -12345
    for extra, off in ((3, 0), (6, 0), (8, 1), (6, 1)):  # scalar, vector, scalar, scalar
        buf = torch.full((m, n + extra), sentinel, dtype=dt, device=x.device)
        y = buf[:, off:off + n]
        P.linear_fwd_prepared(x, wprep, n, fmt, "2:4", y=y, out=out)
        torch.cuda.synchronize()
        b = host(buf)
        got = b[:, off:off + n]
        assert np.array_equal(got.view(np.uint8), ref.view(np.uint8)), f"ldy={n + extra} offset={off}"
        outside = np.concatenate([b[:, :off], b[:, off + n:]], axis=1)
        assert np.all(outside == sentinel), "a store landed outside Y"
