"""Host-side pieces of bench.py (no GPU): the one-GPU contract, and the work and byte
accounting that the TFLOP/s value and the roofline fraction are computed from."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from oracle import resq as oracle  # noqa: E402

KINDS = ["none", "identity", "2:4", "1:4", "4:8", "2:8", "channel50", "channel25",
         "block32x64_50", "block32x64_75", "unstructured50", "unstructured25"]


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("kind", KINDS)
def test_kept_fraction_and_flops_follow_the_oracle_cost_model(kind):
    """The benchmark's FLOP count is the Sec. 5.4 model as the oracle states it."""
    assert bench.kept_fraction(kind) == oracle.kept_fraction(kind)
    for m, d, n in ((256, 2048, 2560), (8192, 18944, 3584), (16, 64, 32)):
        assert bench.alg_flops(m, d, n, kind) == oracle.flops_resq(m, d, n, kind)


def test_flops_of_the_three_named_costs():
    """Sec. 5.4: dense 2mdn; the dense residual doubles it, a 50% residual adds half."""
    m, d, n = 256, 2048, 2560
    assert bench.alg_flops(m, d, n, "none") == 2 * m * d * n
    assert bench.alg_flops(m, d, n, "identity") == 4 * m * d * n
    for kind in ("2:4", "channel50", "block32x64_50", "unstructured50"):
        assert bench.alg_flops(m, d, n, kind) == 3 * m * d * n


def test_bytes_per_element_are_the_formats_storage():
    """4-bit codes plus the block scale: one E8M0 byte per 32 (MXFP4), one 32-bit metadata
    word per 64 (HiF4: 8-bit level-1 code, 8 level-2 and 16 level-3 bits)."""
    assert bench.BYTES_PER_ELEM["mxfp4"] == 0.5 + 1 / 32
    assert bench.BYTES_PER_ELEM["hif4"] == 0.5 + 4 / 64


def test_gemm_bytes_by_hand():
    m, d, n = 16, 64, 32
    # Q(W) + Q(X) + S(Q(dX)) at the format's bytes per element, then fp32 Y
    assert bench.gemm_bytes(m, d, n, "mxfp4", "2:4") == (n * d + 2 * m * d) * 17 / 32 + 4 * m * n
    assert bench.gemm_bytes(m, d, n, "hif4", "2:4") == (n * d + 2 * m * d) * 36 / 64 + 4 * m * n
    # no residual: one activation operand; bf16 output: 2 B per output
    assert bench.gemm_bytes(m, d, n, "mxfp4", "none", y_bytes=2) == (n * d + m * d) * 17 / 32 + 2 * m * n
    # a whole linear: bf16 X in, Q(W) in, Y out
    assert bench.step_bytes(m, d, n, "hif4") == 2 * m * d + n * d * 36 / 64 + 4 * m * n


def test_executed_and_issued_mfma_work():
    """Executed work (the roofline's count): 2mdn per term, the residual dense on gfx950.
    Issued MFMA work: HiF4 runs two MFMAs (hi/lo operands) per term, MXFP4 one."""
    m, d, n = 256, 2048, 2560
    assert bench.executed_flops(m, d, n, "none") == 2 * m * d * n
    assert bench.executed_flops(m, d, n, "2:4") == 4 * m * d * n
    assert bench.executed_flops(m, d, n, "block32x64_50") == 4 * m * d * n
    assert bench.issued_mfma_flops(m, d, n, "mxfp4", "2:4") == 4 * m * d * n
    assert bench.issued_mfma_flops(m, d, n, "hif4", "none") == 4 * m * d * n
    assert bench.issued_mfma_flops(m, d, n, "hif4", "unstructured25") == 8 * m * d * n


def test_extra_entries_cover_the_metric():
    """A default run also measures MXFP4 on the default block, the m = 512 block with each
    global kind, prefill and the backward, each in both formats."""
    names = {(w, f, s) for _, w, f, s in bench.EXTRA_ENTRIES} | {(bench.DEFAULT_WORKLOAD, "hif4", "2:4")}
    for wl in ("qwen3b_layer_m256", "qwen7b_prefill_m8192"):
        assert {(wl, "hif4", "2:4"), (wl, "mxfp4", "2:4")} <= names
    for sp in ("channel50", "block32x64_50", "unstructured50"):
        assert {("qwen7b_layer_m512", f, sp) for f in ("hif4", "mxfp4")} <= names
    assert {("qwen3b_gateup_bwd_m8192", f, "none") for f in ("hif4", "mxfp4")} <= names
    for op in ("w4a16", "w16a4"):
        assert {("qwen3b_layer_m256", f, op) for f in ("hif4", "mxfp4")} <= names
    assert len({k for k, *_ in bench.EXTRA_ENTRIES}) == len(bench.EXTRA_ENTRIES)


def test_traffic_lookup_misses_give_none():
    assert bench.gemm_traffic("no_such_workload", "hif4", "2:4") is None
