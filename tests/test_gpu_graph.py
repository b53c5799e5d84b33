"""HIP graph capture of the entry points (the benchmark times its steps this way): each
replay, with eager calls on the same stream and workspace between the replays, gives the
eager result bit for bit.  Covered: the forward for every residual kind, the backward, the
fused-producer forwards and the mixed-precision linears."""
import pytest

pytestmark = pytest.mark.gpu

# decode shapes: qkv (one K range per workgroup) and down (K split in two, reduction launch)
SHAPES = [(256, 2048, 2560), (256, 11008, 2048)]


def _inputs(torch, m, d, n, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(m, d, generator=g).to(torch.bfloat16).cuda()
    w = (torch.randn(n, d, generator=g) * 0.02).to(torch.bfloat16).cuda()
    return x, w


@pytest.mark.parametrize("sp", ["2:4", "unstructured50", "channel50", "block32x64_50", "none"])
@pytest.mark.parametrize("fmt", ["hif4", "mxfp4"])
@pytest.mark.parametrize("shape", SHAPES, ids=["qkv", "down"])
def test_forward_graph_replays_match_eager(shape, fmt, sp):
    import torch
    import paper_2607_26515_amd as P
    m, d, n = shape
    print(f"graph forward {fmt} {sp} m={m} d={d} n={n}", flush=True)
    x, w = _inputs(torch, m, d, n, 1)
    x_other, _ = _inputs(torch, m, d, n, 2)
    qc, qs = P.quantize(w, fmt, axis=1)
    wp = P.prepare_weights(qc, qs, fmt)
    cs = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(cs):
        ws = P.workspace(P.OP_LINEAR_FWD_PREPARED, P.FORMATS[fmt], P.sparsity_code(sp), m, d, n,
                         x.device)
        y = torch.empty(m, n, dtype=torch.float32, device=x.device)
        y_other = torch.empty_like(y)
        P.linear_fwd_prepared(x, wp, n, fmt, sp, y=y, ws=ws, stream=cs)
        ref = y.clone()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=cs):
            P.linear_fwd_prepared(x, wp, n, fmt, sp, y=y, ws=ws, stream=cs)
        for _ in range(3):
            y.fill_(float("nan"))
            P.linear_fwd_prepared(x_other, wp, n, fmt, sp, y=y_other, ws=ws, stream=cs)
            graph.replay()
            cs.synchronize()
            assert torch.equal(y.view(torch.int32), ref.view(torch.int32))
            assert not torch.equal(y_other.view(torch.int32), ref.view(torch.int32))


@pytest.mark.parametrize("fmt", ["hif4", "mxfp4"])
def test_backward_graph_replays_match_eager(fmt):
    import torch
    import paper_2607_26515_amd as P
    m, d, n = 512, 2048, 2560
    print(f"graph backward {fmt} m={m} d={d} n={n}", flush=True)
    g = torch.Generator().manual_seed(3)
    dy = (torch.randn(m, n, generator=g) * 1e-3).to(torch.bfloat16).cuda()
    dy_other = (torch.randn(m, n, generator=g) * 1e-3).to(torch.bfloat16).cuda()
    x, w = _inputs(torch, m, d, n, 4)
    cs = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(cs):
        ws = P.workspace(P.OP_LINEAR_BWD, P.FORMATS[fmt], P.sparsity_code("none"), m, d, n, x.device)
        dx_ref, dw_ref = P.linear_bwd(dy, x, w, fmt, ws=ws, stream=cs)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=cs):
            dx, dw = P.linear_bwd(dy, x, w, fmt, ws=ws, stream=cs)
        for _ in range(3):
            dx.fill_(float("nan"))
            dw.fill_(float("nan"))
            P.linear_bwd(dy_other, x, w, fmt, ws=ws, stream=cs)
            graph.replay()
            cs.synchronize()
            assert torch.equal(dx.view(torch.int32), dx_ref.view(torch.int32))
            assert torch.equal(dw.view(torch.int32), dw_ref.view(torch.int32))


@pytest.mark.parametrize("producer", ["rmsnorm", "swiglu", "w4a16", "w16a4"])
@pytest.mark.parametrize("fmt", ["hif4", "mxfp4"])
def test_producer_and_mixed_graph_replays_match_eager(fmt, producer):
    """The fused-producer forwards (RMSNorm, SwiGLU) and the mixed-precision linears of
    Table 1 captured in a graph: each replay, with an eager call on other inputs between the
    replays, gives the eager result bit for bit."""
    import torch
    import paper_2607_26515_amd as P
    m, d, n = 256, 2048, 2560
    print(f"graph {producer} {fmt} m={m} d={d} n={n}", flush=True)
    x, w = _inputs(torch, m, d, n, 4)
    x2, _ = _inputs(torch, m, d, n, 5)
    u, _ = _inputs(torch, m, d, n, 6)
    gamma = (1.0 + 0.2 * torch.randn(d, generator=torch.Generator().manual_seed(7))).to(torch.bfloat16).cuda()
    qc, qs = P.quantize(w, fmt, axis=1)
    wp = P.prepare_weights(qc, qs, fmt)
    cs = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(cs):
        if producer == "rmsnorm":
            ws = P.workspace(P.OP_LINEAR_FWD_RMSNORM, P.FORMATS[fmt], P.sparsity_code("2:4"), m, d, n, x.device)
            call = lambda a, y: P.linear_fwd_rmsnorm(a, gamma, 1e-6, wp, n, fmt, "2:4", y=y, ws=ws, stream=cs)
        elif producer == "swiglu":
            ws = P.workspace(P.OP_LINEAR_FWD_PREPARED, P.FORMATS[fmt], P.sparsity_code("2:4"), m, d, n, x.device)
            call = lambda a, y: P.linear_fwd_swiglu(a, u, wp, n, fmt, "2:4", y=y, ws=ws, stream=cs)
        elif producer == "w4a16":
            ws = None
            call = lambda a, y: P.linear_w4a16(a, qc, qs, fmt, y=y, stream=cs)
        else:
            ws = P.workspace(P.OP_LINEAR_W16A4, P.FORMATS[fmt], P.sparsity_code("none"), m, d, n, x.device)
            call = lambda a, y: P.linear_w16a4(a, w, fmt, y=y, ws=ws, stream=cs)
        y = torch.empty(m, n, dtype=torch.float32, device=x.device)
        y_other = torch.empty_like(y)
        call(x, y)
        ref = y.clone()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=cs):
            call(x, y)
        for _ in range(3):
            y.fill_(float("nan"))
            call(x2, y_other)
            graph.replay()
            cs.synchronize()
            assert torch.equal(y.view(torch.int32), ref.view(torch.int32))
            assert not torch.equal(y_other.view(torch.int32), ref.view(torch.int32))
