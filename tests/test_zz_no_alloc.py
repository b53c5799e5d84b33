"""resq_linear_fwd_prepared_noalloc (the forward for callers that cannot allocate) against
resq_linear_fwd_prepared, through the C ABI: same inputs, same Y bit for bit.  Each case
makes two calls in a row on the static scratch, the second with a smaller input, so a value
left behind by the first call (counters, histograms, partial tiles) would show up in the
second.  Oversized calls are rejected before anything is enqueued."""
import numpy as np
import pytest

from synth import WORKLOADS, Linear, Workload, workload_tensors
from _gpu_util import dev_bf16, log

pytestmark = pytest.mark.gpu

# (first call, second call): workload, linear, m of the call (a row prefix of X), sparsity
CASES = [
    # split K (partial tiles in the scratch), then a smaller one-split call
    (("qwen3b_layer_m256", "down", 256, "2:4"), ("qwen3b_layer_m256", "down", 64, "2:4")),
    # element-wise selection (its histogram lives in the scratch), then a smaller one
    (("qwen7b_layer_m512", "qkv", 512, "unstructured50"), ("qwen7b_layer_m512", "qkv", 100, "unstructured50")),
    # block selection, then a smaller channel selection
    (("qwen7b_layer_m512", "o", 512, "block32x64_50"), ("qwen7b_layer_m512", "o", 200, "channel50")),
    # the decode workload's largest linear, then the smallest
    (("qwen3b_layer_m256", "gate_up", 256, "2:4"), ("qwen3b_layer_m256", "qkv", 16, "2:4")),
]


def _inputs(P, fmt, wl_name, lin_name, m):
    wl = WORKLOADS[wl_name]
    lin = next(l for l in wl.linears if l.name == lin_name)
    xb, wb = workload_tensors(wl, lin, seed=0, m=m)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    return dev_bf16(xb), P.prepare_weights(qc, qs, fmt), lin


def _noalloc(P, torch, fmt, sp, x, wprep, n):
    m, d = x.shape
    y = torch.full((m, n), float("nan"), dtype=torch.float32, device=x.device)
    rc = P.resq_linear_fwd_prepared_noalloc(P.FORMATS[fmt], P.sparsity_code(sp), x.data_ptr(), m, d,
                                            x.stride(0), wprep.data_ptr(), n, y.data_ptr(), y.stride(0),
                                            torch.cuda.current_stream().cuda_stream)
    assert rc == 0, P.resq_last_error()
    return y


@pytest.mark.parametrize("fmt", ["hif4", "mxfp4"])
@pytest.mark.parametrize("first,second", CASES)
def test_noalloc_matches_workspace_entry_point(fmt, first, second):
    import torch
    import paper_2607_26515_amd as P
    for wl_name, lin_name, m, sp in (first, second):
        x, wprep, lin = _inputs(P, fmt, wl_name, lin_name, m)
        log(f"noalloc {fmt} {wl_name}/{lin_name} m={m} d={lin.d} n={lin.n} {sp}")
        need = P.resq_workspace_size(P.OP_LINEAR_FWD_PREPARED, P.FORMATS[fmt], P.sparsity_code(sp), m, lin.d, lin.n)
        assert need <= P.NOALLOC_SCRATCH_BYTES
        y = _noalloc(P, torch, fmt, sp, x, wprep, lin.n)
        ref = P.linear_fwd_prepared(x, wprep, lin.n, fmt, sp)
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int32), ref.view(torch.int32)), \
            f"noalloc Y differs from the workspace entry point ({int((y != ref).sum())} outputs)"


def test_noalloc_rejects_sizes_beyond_its_scratch():
    """The m = 8192 prefill down projection needs more than the static scratch: the call
    returns RESQ_ERR_UNSUPPORTED with a message and enqueues nothing (Y keeps its values)."""
    import torch
    import paper_2607_26515_amd as P
    from paper_2607_26515_amd import resq as R
    m, d, n = 8192, 18944, 64
    need = P.resq_workspace_size(P.OP_LINEAR_FWD_PREPARED, P.FORMATS["hif4"], P.sparsity_code("2:4"), m, d, n)
    assert need > P.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((m, d), dtype=torch.int16, device="cuda")
    wprep = torch.zeros(P.resq_prepared_weights_size(P.FORMATS["hif4"], n, d), dtype=torch.uint8, device="cuda")
    y = torch.full((m, n), 7.0, dtype=torch.float32, device="cuda")
    rc = P.resq_linear_fwd_prepared_noalloc(P.FORMATS["hif4"], P.sparsity_code("2:4"), x.data_ptr(), m, d, d,
                                            wprep.data_ptr(), n, y.data_ptr(), n,
                                            torch.cuda.current_stream().cuda_stream)
    assert rc == R.ERR_UNSUPPORTED and "scratch" in P.resq_last_error()
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())
