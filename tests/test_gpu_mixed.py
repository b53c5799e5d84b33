"""GPU parity of the mixed-precision rollout linears (Table 1: W4A16 = X Q(W)^T, W16A4 =
Q(X) W^T) against the oracle.

- Seeded inputs at small ragged sizes (several tiles, ragged edges, a K that ends in half a
  64-chunk for MXFP4), and shapes that take each tile plan (few rows with very many columns,
  few rows with long K, long K with few columns, many column tiles): float32 Y within 1e-5
  normwise of the oracle's float64 result.
- Identity weights, bit for bit: W4A16 with W = c I (Q(c I) = c I) must return c X (the
  activations enter unquantized); W16A4 with W = I must return Q(X), here for every finite
  bf16 value alone in its block.
- The decode workload's linears at full size (m = 256, Qwen2.5-3B), on sampled outputs.
- Operands whose rows lie about 2 GiB apart, which the library splits over several launches
  (the kernel addresses operands with 32-bit offsets)."""
import numpy as np
import pytest

from oracle import formats as F
from oracle import resq as Q
from synth import WORKLOADS, activations, bf16_bits_to_f32, f32_to_bf16_bits, rng_tree, weights, workload_tensors
from _gpu_util import assert_close, dev_bf16, host, log

pytestmark = pytest.mark.gpu

FMTS = ["mxfp4", "hif4"]
C = {"mxfp4": 1.0, "hif4": 1.75}


def _inputs(m, d, n, seed):
    rx, rw = rng_tree(seed, 2)
    return activations(rx, m, d, 0.01, 50.0), weights(rw, n, d)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("m,d,n", [(37, 512, 100), (130, 2048, 700), (256, 1088, 64), (5, 64, 3),
                                   (300, 4096, 520), (5, 64, 65600), (20, 4160, 300), (200, 4096, 96),
                                   (256, 256, 33000), (130, 64, 22000), (20, 128, 20000)])
def test_mixed_forms_match_the_oracle(fmt, m, d, n):
    import paper_2607_26515_amd as P
    if d % F.block_size(fmt):
        pytest.skip("d not a multiple of the block")
    log(f"mixed {fmt} m={m} d={d} n={n}")
    xb, wb = _inputs(m, d, n, m + d + n)
    x, w = bf16_bits_to_f32(xb), bf16_bits_to_f32(wb)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    y4 = host(P.linear_w4a16(dev_bf16(xb), qc, qs, fmt))
    y16 = host(P.linear_w16a4(dev_bf16(xb), dev_bf16(wb), fmt))
    assert_close(y4, Q.w4a16_forward(fmt, x, w)["y64"], f"W4A16 {fmt} {m}x{d}x{n}")
    assert_close(y16, Q.w16a4_forward(fmt, x, w)["y64"], f"W16A4 {fmt} {m}x{d}x{n}")


def test_mxfp4_half_chunk_tail():
    """MXFP4 with d = 96: the last 64-wide K chunk holds one valid 32-block."""
    import paper_2607_26515_amd as P
    xb, wb = _inputs(70, 96, 90, 3)
    x, w = bf16_bits_to_f32(xb), bf16_bits_to_f32(wb)
    qc, qs = P.quantize(dev_bf16(wb), "mxfp4", axis=1)
    assert_close(host(P.linear_w4a16(dev_bf16(xb), qc, qs, "mxfp4")), Q.w4a16_forward("mxfp4", x, w)["y64"])
    assert_close(host(P.linear_w16a4(dev_bf16(xb), dev_bf16(wb), "mxfp4")), Q.w16a4_forward("mxfp4", x, w)["y64"])


def test_operands_beyond_32_bit_offsets():
    """Row strides of about 2 GiB: an operand of three rows then spans more than the kernel's
    32-bit buffer offsets, so the call is split into launches over pieces of the rows of X
    (W4A16) or of W (W16A4)."""
    import torch
    import paper_2607_26515_amd as P
    ld = (1 << 30) - 128  # 2 GiB - 256 bytes per bf16 row: two rows per launch
    m, d, n = 3, 64, 3
    xb, wb = _inputs(m, d, n, 7)
    x, w = bf16_bits_to_f32(xb), bf16_bits_to_f32(wb)
    for fmt in FMTS:
        log(f"mixed 32-bit offset pieces {fmt}")
        big = torch.zeros((m, ld), dtype=torch.int16, device="cuda")
        big[:, :d] = dev_bf16(xb)
        qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
        y4 = host(P.linear_w4a16(big[:, :d], qc, qs, fmt))
        del big
        assert_close(y4, Q.w4a16_forward(fmt, x, w)["y64"], f"W4A16 {fmt}, X rows 2 GiB apart")
        big = torch.zeros((n, ld), dtype=torch.int16, device="cuda")
        big[:, :d] = dev_bf16(wb)
        y16 = host(P.linear_w16a4(dev_bf16(xb), big[:, :d], fmt))
        del big
        torch.cuda.empty_cache()
        assert_close(y16, Q.w16a4_forward(fmt, x, w)["y64"], f"W16A4 {fmt}, W rows 2 GiB apart")


def _finite_bf16():
    b = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    return b[((b >> 7) & 0xFF) != 0xFF]


@pytest.mark.parametrize("fmt", FMTS)
def test_identity_weights_bit_exact(fmt):
    import paper_2607_26515_amd as P
    log(f"mixed identity {fmt}")
    v = _finite_bf16()
    b = F.block_size(fmt)
    xb = np.zeros((v.size, 2 * b), dtype=np.uint16)  # each value alone in its block, twice
    xb[:, 0] = v
    xb[:, 2 * b - 1] = v
    d = 2 * b
    x = bf16_bits_to_f32(xb)
    eye_c = f32_to_bf16_bits(np.eye(d, dtype=np.float32) * np.float32(C[fmt]))
    qc, qs = P.quantize(dev_bf16(eye_c), fmt, axis=1)
    y4 = host(P.linear_w4a16(dev_bf16(xb), qc, qs, fmt))
    # one exact product per output, summed from +0 (so -0 gives +0)
    with np.errstate(over="ignore"):  # 1.75 times the largest bf16 values overflows to inf, as on the GPU
        want4 = (np.float64(C[fmt]) * x.astype(np.float64)).astype(np.float32) + np.float32(0.0)
    assert np.array_equal(y4.view(np.uint32), want4.view(np.uint32)), "W4A16 with W = c I is not c X"
    eye = f32_to_bf16_bits(np.eye(d, dtype=np.float32))
    y16 = host(P.linear_w16a4(dev_bf16(xb), dev_bf16(eye), fmt))
    want16 = F.dequantize(fmt, *F.quantize(fmt, x)).astype(np.float32) + np.float32(0.0)
    assert np.array_equal(y16.view(np.uint32), want16.view(np.uint32)), "W16A4 with W = I is not Q(X)"


@pytest.mark.parametrize("fmt", FMTS)
def test_identity_activations_read_out_every_weight(fmt):
    """W4A16 with X = I returns Q(W)^T itself, so every dequantized weight the GEMM feeds to
    the MFMA is compared bit for bit with the oracle's dequantization of the same codes and
    scales.  Blocks span 2^-33 .. 2^27 in magnitude with elements 1 .. 2^-10 of the block
    maximum, so every scale mantissa, most scale exponents and every level-2 / level-3 shift
    occur."""
    import torch
    import paper_2607_26515_amd as P
    log(f"mixed identity activations {fmt}")
    d, n = 128, 8192
    rng = np.random.default_rng(11)
    b = F.block_size(fmt)
    block_exp = rng.integers(-33, 28, size=(n, d // b, 1)).astype(np.float64)
    mags = np.exp2(block_exp + rng.uniform(-10.0, 0.0, size=(n, d // b, b)))
    w = (mags * rng.choice([-1.0, 1.0], size=mags.shape)).reshape(n, d)
    w[rng.random(w.shape) < 0.05] = 0.0
    wb = f32_to_bf16_bits(w.astype(np.float32))
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    eye = f32_to_bf16_bits(np.eye(d, dtype=np.float32))
    y = host(P.linear_w4a16(dev_bf16(eye), qc, qs, fmt))
    want = F.dequantize(fmt, F.unpack_nibbles(host(qc)), host(qs)).T.astype(np.float32) + np.float32(0.0)
    assert np.array_equal((y + np.float32(0.0)).view(np.uint32), want.view(np.uint32)), "X = I does not give Q(W)^T"


def _samples(rng, size, k):
    idx = set(rng.choice(size, size=min(k, size), replace=False).tolist()) | {0, size - 1}
    return np.array(sorted(idx))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("linear", ["qkv", "o", "gate_up", "down"])
def test_decode_layer_full_size(fmt, linear):
    import torch
    import paper_2607_26515_amd as P
    wl = WORKLOADS["qwen3b_layer_m256"]
    lin = next(l for l in wl.linears if l.name == linear)
    log(f"mixed full-size {wl.name}/{linear} {fmt} m={wl.m} d={lin.d} n={lin.n}")
    xb, wb = workload_tensors(wl, lin, seed=0)
    x, w = dev_bf16(xb), dev_bf16(wb)
    qc, qs = P.quantize(w, fmt, axis=1)
    y4 = P.linear_w4a16(x, qc, qs, fmt)
    y16 = P.linear_w16a4(x, w, fmt)
    torch.cuda.synchronize()
    rng = np.random.default_rng(lin.d + lin.n + 2)
    rows, cols = _samples(rng, wl.m, 12), _samples(rng, lin.n, 48)
    ri, ci = torch.as_tensor(rows, device=x.device), torch.as_tensor(cols, device=x.device)
    xs, ws = bf16_bits_to_f32(xb[rows]), bf16_bits_to_f32(wb[cols])
    assert_close(host(y4[ri][:, ci]), Q.w4a16_forward(fmt, xs, ws)["y64"], f"W4A16 {linear} {fmt}")
    assert_close(host(y16[ri][:, ci]), Q.w16a4_forward(fmt, xs, ws)["y64"], f"W16A4 {linear} {fmt}")
