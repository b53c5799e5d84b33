"""The synthetic-input module: its bf16 rounding and its seeding (no arithmetic of the method
lives there)."""
import numpy as np

from synth import WORKLOADS, bf16_bits_to_f32, f32_to_bf16_bits, workload_tensors


def test_bf16_rounding_matches_torch_on_edge_and_random_values():
    """Nearest-even float32 -> bf16 rounding, against torch's conversion: the largest finite
    values of both signs, subnormals, exact midpoints and two million random bit patterns."""
    import torch
    rng = np.random.default_rng(0)
    pats = rng.integers(0, 1 << 32, size=2_000_000, dtype=np.uint64).astype(np.uint32)
    edge = np.array([0x7F7FFFFF, 0xFF7FFFFF, 0x00000001, 0x80000001, 0x007FFFFF, 0x00008000,
                     0x00018000, 0x3F808000, 0x3F818000, 0x7F7F8000, 0x00000000, 0x80000000],
                    dtype=np.uint32)
    u = np.concatenate([pats, edge])
    u = u[((u >> 23) & 0xFF) != 0xFF]  # finite only
    x = u.view(np.float32)
    want = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(f32_to_bf16_bits(x), want)


def test_widening_is_exact():
    b = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    b = b[((b >> 7) & 0xFF) != 0xFF]
    assert np.array_equal(f32_to_bf16_bits(bf16_bits_to_f32(b)), b)


def test_row_prefix_of_a_workload_is_the_same_draw():
    """Asking for fewer rows gives the first rows of the full draw (samples of the benchmark
    inputs are the inputs' own rows)."""
    wl = WORKLOADS["single_m16"]
    lin = wl.linears[0]
    x, w = workload_tensors(wl, lin)
    x4, w4 = workload_tensors(wl, lin, m=4)
    assert np.array_equal(x4, x[:4]) and np.array_equal(w4, w)
    x5, w5 = workload_tensors(wl, lin, m=5, n_w=7)
    assert np.array_equal(x5, x[:5]) and np.array_equal(w5, w[:7])
