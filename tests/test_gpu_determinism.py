"""Run-to-run determinism of every GEMM plan, bit for bit.

The GEMM sums each output in a fixed order (no atomics; K groups and K splits are added in
group and split order), so two calls with identical inputs must give identical bits.  A
stage-protocol race (a copy still in flight when its LDS stage is read, or a stage refilled
while another wave still reads it) would show up as a difference between the two calls.
The cases below run each tile configuration, K-group count, stage count and K split that
launch_gemm instantiates (the CPU test at the bottom checks that, from the host-side plan
query), at the benchmark shapes, the prefill ones included."""
import numpy as np
import pytest

from synth import WORKLOADS, Workload, Linear, workload_tensors
from _gpu_util import dev_bf16, log

# (workload, linear, sparsity) forward cases; sizes are the benchmark workloads' own, plus
# the 7B down projection at m = 256
_EXTRA = Workload("qwen7b_down_m256", 256, (Linear("down", 18944, 3584),), 0.005, 100.0)
# backward cases: the training workload, a narrow one whose dW GEMM (256 x 256 over
# K = 8192, not split) takes the small tiles with four K groups and four stages (MXFP4), and
# a square one whose dW GEMM (1536 x 1536 over K = 8192, not split) fills more than the CUs
# with them (MXFP4: four K groups, two stages; HiF4: two and two)
_NARROW_BWD = Workload("narrow_bwd_m8192", 8192, (Linear("proj", 256, 256),), 0.01, 50.0, backward=True)
_SQUARE_BWD = Workload("square_bwd_m8192", 8192, (Linear("proj", 1536, 1536),), 0.01, 50.0, backward=True)
BWD_CASES = ["qwen3b_gateup_bwd_m8192", "narrow_bwd_m8192", "square_bwd_m8192"]
FWD_CASES = [
    ("qwen3b_layer_m256", "qkv", "2:4"),
    ("qwen3b_layer_m256", "qkv", "none"),
    ("qwen3b_layer_m256", "gate_up", "2:4"),
    ("qwen3b_layer_m256", "down", "2:4"),
    ("qwen7b_layer_m512", "qkv", "unstructured50"),
    ("qwen7b_layer_m512", "down", "block32x64_50"),
    ("qwen7b_layer_m512", "gate_up", "channel50"),
    ("qwen7b_down_m256", "down", "2:4"),
    ("qwen7b_prefill_m8192", "down", "2:4"),
    ("qwen7b_prefill_m8192", "gate_up", "2:4"),
    ("qwen7b_prefill_m8192", "gate_up", "none"),
]
FMTS = ["mxfp4", "hif4"]


def _workload(name):
    return {_EXTRA.name: _EXTRA, _NARROW_BWD.name: _NARROW_BWD, _SQUARE_BWD.name: _SQUARE_BWD}.get(name) or WORKLOADS[name]


def _plan_key(P, fmt, M, N, K, split):
    p = P.gemm_plan(fmt, M, N, K, split)
    return (fmt, p["tile"], p["kgroups"], p["stages"], p["ksplit"] > 1)


# every (format, tile, K groups, stages, K split) that launch_gemm can run
INSTANTIATED = {
    ("mxfp4", "64x64", 2, 4, False), ("mxfp4", "64x64", 4, 4, False), ("mxfp4", "64x64", 4, 2, False),
    ("mxfp4", "64x64", 1, 4, False), ("mxfp4", "128x256", 1, 4, False), ("mxfp4", "128x256", 1, 4, True),
    ("mxfp4", "64x128", 1, 4, True), ("mxfp4", "64x128", 1, 4, False),
    ("hif4", "64x64", 2, 4, False), ("hif4", "64x64", 2, 2, False), ("hif4", "64x64", 1, 2, False),
    ("hif4", "128x192_8w", 1, 2, False), ("hif4", "128x192", 1, 2, False), ("hif4", "128x192", 1, 2, True),
    ("hif4", "64x128", 2, 2, True),
}


def test_cases_cover_every_plan():
    """CPU: the forward and backward cases of this file run every instantiated GEMM plan."""
    import paper_2607_26515_amd as P
    seen = set()
    for fmt in FMTS:
        for wl_name, lin_name, _ in FWD_CASES:
            wl = _workload(wl_name)
            lin = next(l for l in wl.linears if l.name == lin_name)
            seen.add(_plan_key(P, fmt, wl.m, lin.n, lin.d, True))
        for name in BWD_CASES:
            wl = _workload(name)
            lin = wl.linears[0]
            seen.add(_plan_key(P, fmt, wl.m, lin.d, lin.n, False))  # dX
            seen.add(_plan_key(P, fmt, lin.n, lin.d, wl.m, False))  # dW
    assert seen <= INSTANTIATED, f"unexpected plans {seen - INSTANTIATED}"
    assert INSTANTIATED <= seen, f"plans not covered: {INSTANTIATED - seen}"


def _same_bits(a, b):
    import torch
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


@pytest.mark.gpu
@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("wl_name,lin_name,sp", FWD_CASES)
def test_forward_twice_same_bits(fmt, wl_name, lin_name, sp):
    import torch
    import paper_2607_26515_amd as P
    wl = _workload(wl_name)
    lin = next(l for l in wl.linears if l.name == lin_name)
    plan = P.gemm_plan(fmt, wl.m, lin.n, lin.d, True)
    log(f"determinism fwd {wl_name}/{lin_name} {fmt} {sp} m={wl.m} d={lin.d} n={lin.n} plan={plan}")
    xb, wb = workload_tensors(wl, lin, seed=0)
    x = dev_bf16(xb)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    wprep = P.prepare_weights(qc, qs, fmt)
    del qc, qs
    ws = P.workspace(P.OP_LINEAR_FWD_PREPARED, fmt, P.sparsity_code(sp), wl.m, lin.d, lin.n, x.device)
    y1 = P.linear_fwd_prepared(x, wprep, lin.n, fmt, sp, ws=ws)
    y2 = P.linear_fwd_prepared(x, wprep, lin.n, fmt, sp, ws=ws)
    torch.cuda.synchronize()
    assert _same_bits(y1, y2), f"two identical calls differ ({int((y1 != y2).sum())} outputs)"


@pytest.mark.gpu
@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("name", BWD_CASES)
def test_backward_twice_same_bits(fmt, name):
    import torch
    import paper_2607_26515_amd as P
    wl = _workload(name)
    lin = wl.linears[0]
    log(f"determinism bwd {wl.name} {fmt} m={wl.m} d={lin.d} n={lin.n}")
    xb, wb, gb = workload_tensors(wl, lin, seed=0)
    g, x, w = dev_bf16(gb), dev_bf16(xb), dev_bf16(wb)
    dx1, dw1 = P.linear_bwd(g, x, w, fmt)
    dx2, dw2 = P.linear_bwd(g, x, w, fmt)
    torch.cuda.synchronize()
    assert _same_bits(dx1, dx2), "dX differs between two identical calls"
    assert _same_bits(dw1, dw2), "dW differs between two identical calls"


_SPLIT_CASES = [("qwen3b_layer_m256", "down", "2:4"), ("qwen7b_down_m256", "down", "2:4"),
                ("qwen7b_layer_m512", "down", "block32x64_50"), ("qwen7b_layer_m512", "down", "unstructured50")]


@pytest.mark.gpu
@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("wl_name,lin_name,sp", _SPLIT_CASES)
def test_split_k_from_any_workspace(fmt, wl_name, lin_name, sp):
    """A K-split GEMM keeps its partial tiles in the workspace, and every partial is written
    before the reduction reads it: a workspace full of 0xFF bytes, the same workspace used
    again, and a zeroed one give the same bits."""
    import torch
    import paper_2607_26515_amd as P
    wl = _workload(wl_name)
    lin = next(l for l in wl.linears if l.name == lin_name)
    plan = P.gemm_plan(fmt, wl.m, lin.n, lin.d, True)
    log(f"split-K workspace {wl_name}/{lin_name} {fmt} {sp} plan={plan}")
    assert plan["ksplit"] > 1, "the case must split K"
    xb, wb = workload_tensors(wl, lin, seed=1)
    x = dev_bf16(xb)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    wprep = P.prepare_weights(qc, qs, fmt)
    del qc, qs
    code = P.sparsity_code(sp)
    dirty = P.workspace(P.OP_LINEAR_FWD_PREPARED, fmt, code, wl.m, lin.d, lin.n, x.device)
    dirty[0].fill_(255)
    clean = P.workspace(P.OP_LINEAR_FWD_PREPARED, fmt, code, wl.m, lin.d, lin.n, x.device)
    clean[0].zero_()
    y1 = P.linear_fwd_prepared(x, wprep, lin.n, fmt, sp, ws=dirty)
    y2 = P.linear_fwd_prepared(x, wprep, lin.n, fmt, sp, ws=dirty)
    y3 = P.linear_fwd_prepared(x, wprep, lin.n, fmt, sp, ws=clean)
    torch.cuda.synchronize()
    assert _same_bits(y1, y3), f"dirty workspace: {int((y1 != y3).sum())} outputs differ"
    assert _same_bits(y2, y3), f"reused workspace: {int((y2 != y3).sum())} outputs differ"
