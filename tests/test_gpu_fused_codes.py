"""The residual operand the forward GEMM consumes, bit for bit (Sec. 4.3, Eq. 4).

resq_linear_fwd_prepared writes S(Q(dX)) as MFMA fragments inside its own activation pass
(local kinds) or its selection pass (channel, block and element-wise kinds); these are not the
kernels resq_residual_sparsify runs, whose masks other tests compare.  With W = c I (n = d;
c = 1 for MXFP4 and 1.75 for HiF4, both represented exactly by Q), output (i, j) holds one
main product c Q(X)[i, j] and one residual product c S(Q(dX))[i, j] (every other product is
an exact zero).  For these inputs each such sum is exact in float32 (the test checks that
with the oracle), so Y must equal the oracle's c (Q(X) + S(Q(dX))) bit for bit: a mis-kept,
mis-pruned or mis-quantized residual element changes Y.  Kept elements that quantize to
zero and pruned ones both give 0; the values, which are unique, are what is compared.
The fused SwiGLU producer's X (reading F1) is checked the same way."""
import numpy as np
import pytest

from oracle import formats as F
from oracle import resq as Q
from synth import WORKLOADS, activations, bf16_bits_to_f32, f32_to_bf16_bits, rng_tree, workload_tensors
from _gpu_util import dev_bf16, host, log

pytestmark = pytest.mark.gpu

FMTS = ["mxfp4", "hif4"]
C = {"mxfp4": 1.0, "hif4": 1.75}
KINDS = ["2:4", "1:4", "4:8", "channel50", "block32x64_50", "unstructured50"]
SHAPES = [("qwen3b_layer_m256", "qkv"), ("qwen7b_layer_m512", "qkv")]  # m=256 d=2048; m=512 d=3584


def _identity_prepared(P, fmt, d):
    c = np.float32(C[fmt])
    w = np.eye(d, dtype=np.float32) * c
    assert np.array_equal(F.dequantize(fmt, *F.quantize(fmt, w[:64])), w[:64]), "Q(c I) != c I"
    qc, qs = P.quantize(dev_bf16(f32_to_bf16_bits(w)), fmt, axis=1)
    return P.prepare_weights(qc, qs, fmt)


def _expected(fmt, sp, x):
    o = Q.resq_quantize_residual(fmt, sp, x)
    c = float(C[fmt])
    exact = c * o["xhat"].astype(np.float64)
    if sp != "none":
        exact = exact + c * o["srhat"].astype(np.float64)
    want = exact.astype(np.float32)
    assert np.array_equal(want.astype(np.float64), exact), "a sum is not exact in float32"
    return want + np.float32(0.0)  # the GEMM's sums start from +0: -0 becomes +0


def _check(y, want, what):
    if not np.array_equal(y.view(np.uint32), want.view(np.uint32)):
        bad = np.argwhere(y.view(np.uint32) != want.view(np.uint32))
        i, j = bad[0]
        raise AssertionError(f"{what}: {len(bad)} elements of c (Q(X) + S(Q(dX))) differ, first "
                             f"({i}, {j}): {y[i, j]!r} vs {want[i, j]!r}")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", KINDS)
@pytest.mark.parametrize("wl_name,lin_name", SHAPES)
def test_forward_residual_operand_bits(fmt, sp, wl_name, lin_name):
    import paper_2607_26515_amd as P
    wl = WORKLOADS[wl_name]
    lin = next(l for l in wl.linears if l.name == lin_name)
    m, d = wl.m, lin.d
    log(f"fused residual operand {wl_name}/{lin_name} X, {fmt} {sp} m={m} d={d} (W = c I)")
    xb, _ = workload_tensors(wl, lin, seed=0)
    y = host(P.linear_fwd_prepared(dev_bf16(xb), _identity_prepared(P, fmt, d), d, fmt, sp))
    _check(y, _expected(fmt, sp, bf16_bits_to_f32(xb)), f"{wl_name} {fmt} {sp}")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("sp", ["none", "2:4", "unstructured50"])
def test_swiglu_operands_bits(fmt, sp):
    """The fused SwiGLU producer: X = silu(G) U is formed inside the activation pass; Q(X)
    and S(Q(dX)) as the GEMM consumes them equal the oracle's for the oracle's X."""
    import paper_2607_26515_amd as P
    m, d = 256, 2048
    log(f"fused swiglu operands {fmt} {sp} m={m} d={d} (W = c I)")
    rg, ru = rng_tree(11, 2)
    gb, ub = activations(rg, m, d, 0.01, 8.0), activations(ru, m, d, 0.01, 30.0)
    y = host(P.linear_fwd_swiglu(dev_bf16(gb), dev_bf16(ub), _identity_prepared(P, fmt, d), d, fmt, sp))
    xb = Q.swiglu_bf16(bf16_bits_to_f32(gb), bf16_bits_to_f32(ub))
    _check(y, _expected(fmt, sp, bf16_bits_to_f32(xb)), f"swiglu {fmt} {sp}")
