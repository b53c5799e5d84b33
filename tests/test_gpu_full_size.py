"""GPU <-> oracle parity at the full sizes of the benchmark workloads, on sampled outputs.

The GPU runs each linear at its real shape through the same entry point bench.py times
(resq_linear_fwd_prepared, or resq_linear_bwd).  The oracle then computes a sample of
outputs one by one.
- Forward with local residual kinds: every row of Y depends on its own row of X and on
  rows of Q(W), so a sample of (row, column) pairs needs only those rows quantized.
- Forward with global kinds: the selection of S(Q(dX)) is computed over the whole tensor.
- Backward: dX[i, c] needs row i of dY and column c of W, each quantized along n; dW[j, c]
  needs columns j of dY and c of X, each quantized along m.
Tolerance: normwise relative error of the sampled outputs <= 1e-5."""
import numpy as np
import pytest

from oracle import formats as F
from oracle import resq as Q
from synth import WORKLOADS, bf16_bits_to_f32, workload_tensors
from _gpu_util import Y_TOL, assert_close, dev_bf16, host, log

pytestmark = pytest.mark.gpu

FMTS = ["hif4", "mxfp4"]


def _samples(rng, size, k):
    """k random indices plus both ends (covers the ragged last tile)."""
    idx = set(rng.choice(size, size=min(k, size), replace=False).tolist()) | {0, size - 1}
    return np.array(sorted(idx))


def _wrows(fmt, wb, cols):
    """Dequantized Q(W) rows (blocks along d) for the sampled output features."""
    w = bf16_bits_to_f32(wb[cols])
    return F.dequantize(fmt, *F.quantize(fmt, w))


def _fwd_full(fmt, sp, wl_name, lin_name, n_rows=12, n_cols=48, out="f32"):
    import torch
    import paper_2607_26515_amd as P
    wl = WORKLOADS[wl_name]
    lin = next(l for l in wl.linears if l.name == lin_name)
    log(f"full-size fwd {wl_name}/{lin_name} {fmt} {sp} {out} m={wl.m} d={lin.d} n={lin.n}")
    xb, wb = workload_tensors(wl, lin, seed=0)
    x = dev_bf16(xb)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    wprep = P.prepare_weights(qc, qs, fmt)
    del qc, qs
    y = P.linear_fwd_prepared(x, wprep, lin.n, fmt, sp)
    if out == "bf16":
        # the bf16 entry point: its output is the bf16 rounding of the float32 one, everywhere
        yb = P.linear_fwd_prepared(x, wprep, lin.n, fmt, sp, out="bf16")
        torch.cuda.synchronize()
        assert torch.equal(yb, y.to(torch.bfloat16).view(torch.int16)), "bf16 Y != bf16(float32 Y)"
        del yb
    torch.cuda.synchronize()
    rng = np.random.default_rng(lin.d + lin.n)
    rows, cols = _samples(rng, wl.m, n_rows), _samples(rng, lin.n, n_cols)
    ys = host(y[torch.as_tensor(rows, device=y.device)][:, torch.as_tensor(cols, device=y.device)])
    del y, wprep, x
    if Q.parse_sparsity(sp)[0] in ("channel", "block", "unstructured"):
        o = Q.resq_quantize_residual(fmt, sp, bf16_bits_to_f32(xb))  # global selection
        a = o["xhat"][rows].astype(np.float64) + o["srhat"][rows]
    else:
        o = Q.resq_quantize_residual(fmt, sp, bf16_bits_to_f32(xb[rows]))
        a = o["xhat"].astype(np.float64) + (o["srhat"] if sp != "none" else 0.0)
    want = a @ _wrows(fmt, wb, cols).T
    return assert_close(ys, want, f"Y sample {wl_name}/{lin_name} {fmt} {sp}")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("linear", ["qkv", "o", "gate_up", "down"])
def test_qwen3b_layer_m256_full(fmt, linear):
    """The bench workload: every linear of the Qwen2.5-3B block at m = 256, S_2:4."""
    _fwd_full(fmt, "2:4", "qwen3b_layer_m256", linear)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["unstructured50", "block32x64_50", "channel50"])
@pytest.mark.parametrize("linear", ["qkv", "o", "gate_up", "down"])
def test_qwen7b_layer_m512_full(fmt, sp, linear):
    _fwd_full(fmt, sp, "qwen7b_layer_m512", linear)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("linear", ["gate_up", "down"])
def test_qwen3b_layer_m256_bf16_out_full(fmt, linear):
    """The bench's --out bf16 line: bf16 Y equals the rounding of the float32 Y everywhere,
    and the float32 Y matches the oracle on the sample."""
    _fwd_full(fmt, "2:4", "qwen3b_layer_m256", linear, out="bf16")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["unstructured25", "channel75", "block32x64_25", "4:8", "1:4"])
def test_qwen7b_layer_m512_levels_full(fmt, sp):
    """Other sparsity levels and k:g patterns at the m = 512 block's qkv shape."""
    _fwd_full(fmt, sp, "qwen7b_layer_m512", "qkv")


def _swiglu_full(fmt, wl_name, n_rows, n_cols):
    """The down projection with its SwiGLU input fused (bench --op swiglu_down), G and U
    drawn as the benchmark draws them; the oracle forms X for the sampled rows only."""
    import torch
    import paper_2607_26515_amd as P
    from synth import activations, rng_tree
    wl = WORKLOADS[wl_name]
    lin = next(l for l in wl.linears if l.name == "down")
    m, d, n = wl.m, lin.d, lin.n
    log(f"full-size swiglu down {wl_name} {fmt} m={m} d={d} n={n}")
    _, wb = workload_tensors(wl, lin, seed=0)
    rg, ru = rng_tree(7, 2)
    gb, ub = activations(rg, m, d, 0.01, 8.0), activations(ru, m, d, 0.01, 30.0)
    qc, qs = P.quantize(dev_bf16(wb), fmt, axis=1)
    wprep = P.prepare_weights(qc, qs, fmt)
    del qc, qs
    y = P.linear_fwd_swiglu(dev_bf16(gb), dev_bf16(ub), wprep, n, fmt, "2:4")
    torch.cuda.synchronize()
    rng = np.random.default_rng(d + n + 1)
    rows, cols = _samples(rng, m, n_rows), _samples(rng, n, n_cols)
    ys = host(y[torch.as_tensor(rows, device=y.device)][:, torch.as_tensor(cols, device=y.device)])
    del y, wprep
    xs = Q.swiglu_bf16(bf16_bits_to_f32(gb[rows]), bf16_bits_to_f32(ub[rows]))
    o = Q.resq_quantize_residual(fmt, "2:4", bf16_bits_to_f32(xs))
    want = (o["xhat"].astype(np.float64) + o["srhat"]) @ _wrows(fmt, wb, cols).T
    assert_close(ys, want, f"Y sample swiglu {wl_name} {fmt}")


@pytest.mark.parametrize("fmt", FMTS)
def test_qwen3b_swiglu_down_m256_full(fmt):
    _swiglu_full(fmt, "qwen3b_layer_m256", 12, 48)


@pytest.mark.parametrize("fmt", FMTS)
def test_qwen7b_swiglu_down_m8192_full(fmt):
    _swiglu_full(fmt, "qwen7b_prefill_m8192", 8, 32)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("linear", ["down", "gate_up"])
def test_qwen7b_prefill_m8192_full(fmt, linear):
    _fwd_full(fmt, "2:4", "qwen7b_prefill_m8192", linear, n_rows=8, n_cols=32)


def _col_quant(fmt, v):
    """Dequantized Q of a vector quantized in blocks along its length."""
    return F.dequantize(fmt, *F.quantize(fmt, v[None, :].astype(np.float32)))[0]


@pytest.mark.parametrize("fmt", FMTS)
def test_qwen3b_gateup_bwd_m8192_full(fmt):
    import torch
    import paper_2607_26515_amd as P
    wl = WORKLOADS["qwen3b_gateup_bwd_m8192"]
    lin = wl.linears[0]
    m, d, n = wl.m, lin.d, lin.n
    log(f"full-size bwd {fmt} m={m} d={d} n={n}")
    xb, wb, gb = workload_tensors(wl, lin, seed=0)
    dx, dw = P.linear_bwd(dev_bf16(gb), dev_bf16(xb), dev_bf16(wb), fmt)
    torch.cuda.synchronize()
    rng = np.random.default_rng(7)
    ri, cd, rn = _samples(rng, m, 6), _samples(rng, d, 12), _samples(rng, n, 6)
    dxs = host(dx[torch.as_tensor(ri, device=dx.device)][:, torch.as_tensor(cd, device=dx.device)])
    dws = host(dw[torch.as_tensor(rn, device=dw.device)][:, torch.as_tensor(cd, device=dw.device)])
    del dx, dw
    gy, x, w = bf16_bits_to_f32(gb), bf16_bits_to_f32(xb), bf16_bits_to_f32(wb)
    # dX[i, c] = Q_n(dY)[i, :] . Q_n(W)[:, c]
    qdy_rows = F.dequantize(fmt, *F.quantize(fmt, gy[ri]))
    qw_cols = np.stack([_col_quant(fmt, w[:, c]) for c in cd], axis=1)
    assert_close(dxs, qdy_rows @ qw_cols, f"dX sample {fmt}")
    # dW[j, c] = Q_m(dY)[:, j] . Q_m(X)[:, c]
    qdy_cols = np.stack([_col_quant(fmt, gy[:, j]) for j in rn], axis=1)
    qx_cols = np.stack([_col_quant(fmt, x[:, c]) for c in cd], axis=1)
    assert_close(dws, qdy_cols.T @ qx_cols, f"dW sample {fmt}")
    assert Y_TOL == 1e-5
