"""Global selections beyond the register-resident top-k (more than 20,480 channels or
blocks), where each radix pass streams the keys: S^{32x64}_50% at the prefill down
projection's size (m = 8192, d = 18944: 75,776 blocks), S_50% over 32,768 channels, and the
element-wise kind over enough workgroups to span several tie-count groups.

The oracle's Q(dX) is row-local, so it is evaluated in row chunks (multiples of 32 rows, so
each 32 x 64 block lies in one chunk); the block keys of all chunks are then ranked together
by the oracle's top-k.  That is the oracle's block selection (Sec. 4.3) evaluated piecewise,
with the same functions and the same summation order."""
import numpy as np
import pytest

from oracle import resq as Q
from synth import WORKLOADS, activations, bf16_bits_to_f32, rng_tree, workload_tensors
from _gpu_util import assert_close, dev_bf16, host, log, pack_bits

pytestmark = pytest.mark.gpu

CHUNK = 1024  # rows per oracle chunk (a multiple of 32)


def _oracle_block_mask(fmt, xb, pct=50):
    """Kept 32 x 64 blocks (ceil(m/32), d/64) and the per-chunk Q(X), Q(dX) on demand."""
    m, d = xb.shape
    keys = []
    for r0 in range(0, m, CHUNK):
        o = Q.resq_quantize_residual(fmt, "identity", bf16_bits_to_f32(xb[r0:r0 + CHUNK]))
        keys.append(Q.block_keys(o["srhat"], fmt))
    keys = np.concatenate(keys, axis=0)
    return Q._top(keys.ravel(), pct).reshape(keys.shape)


@pytest.mark.parametrize("fmt", ["hif4", "mxfp4"])
def test_block_selection_prefill_down_full_size(fmt):
    """resq_residual_sparsify's block mask and the forward's Y (sampled) at m = 8192,
    d = 18944, the prefill workload's own X."""
    import torch
    import paper_2607_26515_amd as P
    wl = WORKLOADS["qwen7b_prefill_m8192"]
    lin = wl.linears[0]
    m, d, n = wl.m, lin.d, lin.n
    log(f"large block selection {fmt} m={m} d={d} ({((m + 31) // 32) * (d // 64)} blocks)")
    xb, wb = workload_tensors(wl, lin, seed=0)
    x = dev_bf16(xb)
    out = P.residual_sparsify(x, fmt, "block32x64_50")
    got = host(out["group_mask"])
    del out
    blk = _oracle_block_mask(fmt, xb)
    want = pack_bits(blk.ravel())
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        raise AssertionError(f"block mask: {len(bad)} bytes differ, first at {bad[:5].tolist()}")
    assert int(np.unpackbits(got, bitorder="little").sum()) == blk.size // 2
    # the forward with the same selection, sampled rows and columns against the oracle
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    y = P.linear_fwd_prepared(x, P.prepare_weights(qc, qs, fmt), n, fmt, "block32x64_50")
    torch.cuda.synchronize()
    rng = np.random.default_rng(7)
    rows = np.array(sorted(set(rng.choice(m, 10, replace=False).tolist()) | {0, m - 1}))
    cols = np.array(sorted(set(rng.choice(n, 40, replace=False).tolist()) | {0, n - 1}))
    ys = host(y[torch.as_tensor(rows, device=y.device)][:, torch.as_tensor(cols, device=y.device)])
    del y, x
    o = Q.resq_quantize_residual(fmt, "identity", bf16_bits_to_f32(xb[rows]))
    keep = np.repeat(blk[rows // 32], 64, axis=1)  # the kept blocks of the sampled rows
    a = o["xhat"].astype(np.float64) + np.where(keep, o["srhat"], 0.0)
    w = bf16_bits_to_f32(wb[cols])
    from oracle import formats as F
    what = F.dequantize(fmt, *F.quantize(fmt, w))
    assert_close(ys, a @ what.T.astype(np.float64), f"Y sample, block selection {fmt} m={m} d={d}")


@pytest.mark.parametrize("fmt", ["hif4", "mxfp4"])
@pytest.mark.parametrize("d", [20480, 20544, 32768])
def test_channel_selection_at_and_beyond_the_register_limit(fmt, d):
    """20,480 channels fill the top-k's registers (20 keys per thread); 20,544 and 32,768 take
    the streaming top-k."""
    import paper_2607_26515_amd as P
    m = 64
    log(f"large channel selection {fmt} m={m} d={d}")
    xb = activations(rng_tree(21, 1)[0], m, d, 0.01, 50.0)
    out = P.residual_sparsify(dev_bf16(xb), fmt, "channel50")
    o = Q.resq_quantize_residual(fmt, "channel50", bf16_bits_to_f32(xb))
    assert np.array_equal(host(out["group_mask"]), pack_bits(o["groups"].ravel())), "channel mask"
    assert np.array_equal(host(out["keep_mask"]), pack_bits(o["keep"])), "keep mask"


@pytest.mark.parametrize("fmt", ["hif4", "mxfp4"])
def test_element_selection_many_tie_groups(fmt):
    """2048 x 4096: 1024 workgroups in the element-wise passes (four tie-count groups), with
    most keys tied (a representable half of the tensor gives exact zeros)."""
    import paper_2607_26515_amd as P
    m, d = 2048, 4096
    log(f"element selection, many tie groups {fmt} m={m} d={d}")
    xb = activations(rng_tree(22, 1)[0], m, d, 0.01, 50.0)
    xb[: m // 2] &= np.uint16(0xFF80)  # keep only the sign and exponent: many exact values, Q(dX) ties
    out = P.residual_sparsify(dev_bf16(xb), fmt, "unstructured50")
    o = Q.resq_quantize_residual(fmt, "unstructured50", bf16_bits_to_f32(xb))
    assert np.array_equal(host(out["keep_mask"]), pack_bits(o["keep"])), "keep mask"
