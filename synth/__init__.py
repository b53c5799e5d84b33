"""Seeded synthetic inputs for the Rollout-ResQ linear layer.

This module is shared by the tests, the benchmark and the oracle's test harness.  It holds
none of the method's arithmetic: it only draws arrays with numpy's PCG64 generator, scales a
seeded subset of input channels to mimic the activation outliers that the paper identifies as
the cause of FP4 zero collapse (Sec. 4.2, Fig. 2), and rounds float32 draws to bfloat16.

bfloat16 arrays are carried as ``uint16`` bit patterns (numpy has no bf16 dtype).

Workloads (the shapes of the paper's Qwen2.5-3B / Qwen2.5-Math-7B linear projections,
Sec. 5.1; the paper's own activations and weights are not available, so seeded synthetic
tensors with the same shapes and outlier structure stand in for them):

* ``single_m16``      one linear, m=16, d=2048 -> n=2048
* ``qwen3b_layer_m256``  the four linears of one Qwen2.5-3B block at m=256 tokens
* ``qwen7b_layer_m512``  the four linears of one Qwen2.5-Math-7B block at m=512 tokens
* ``qwen7b_prefill_m8192`` 7B down_proj and gate_up at m=8192 tokens (Student-t nu=3 + outliers)
* ``qwen3b_gateup_bwd_m8192`` backward of the 3B gate_up projection at m=8192
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Tuple

import numpy as np

__all__ = [
    "f32_to_bf16_bits",
    "bf16_bits_to_f32",
    "rng_tree",
    "activations",
    "weights",
    "grad_output",
    "Linear",
    "Workload",
    "WORKLOADS",
    "workload_tensors",
]


# ----------------------------------------------------------------------------------------
# bfloat16 <-> float32 (bit-pattern helpers; rounding of the synthetic draws only)
# ----------------------------------------------------------------------------------------
def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16, nearest-even, and return the uint16 bit patterns.

    Inputs must be finite (the generators never produce NaN or Inf).
    """
    # for a finite float32 the sum below stays under 2^32 (the largest pattern, 0xFF7FFFFF,
    # plus 0x8000), so 32-bit arithmetic is exact
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = u + np.uint32(0x7FFF)
    r += (u >> 16) & np.uint32(1)
    r >>= 16
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ----------------------------------------------------------------------------------------
# generators
# ----------------------------------------------------------------------------------------
def rng_tree(seed: int, n: int) -> List[np.random.Generator]:
    """``n`` independent PCG64 streams derived from one seed (one per tensor)."""
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(n)]


def activations(rng: np.random.Generator, m: int, d: int, outlier_frac: float,
                outlier_scale: float, dist: str = "normal") -> np.ndarray:
    """bf16 activations ``m x d``: N(0,1) (or Student-t nu=3) with outlier channels.

    ``round(outlier_frac * d)`` input channels (columns), drawn without replacement, are
    multiplied by ``outlier_scale``.
    """
    # the outlier channels are drawn first so that they do not depend on m
    n_out = int(round(outlier_frac * d))
    cols = rng.choice(d, size=n_out, replace=False) if n_out > 0 else np.zeros(0, np.int64)
    if dist == "normal":
        x = rng.standard_normal((m, d), dtype=np.float32)
    elif dist == "t3":
        x = rng.standard_t(3.0, size=(m, d)).astype(np.float32)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    if n_out > 0:
        x[:, cols] *= np.float32(outlier_scale)
    return f32_to_bf16_bits(x)


def weights(rng: np.random.Generator, n: int, d: int, std: float = 0.02) -> np.ndarray:
    """bf16 weights ``n x d`` drawn from N(0, std)."""
    return f32_to_bf16_bits(rng.standard_normal((n, d), dtype=np.float32) * np.float32(std))


def grad_output(rng: np.random.Generator, m: int, n: int, std: float = 1e-3) -> np.ndarray:
    """bf16 output gradient ``m x n`` drawn from N(0, std)."""
    return f32_to_bf16_bits(rng.standard_normal((m, n), dtype=np.float32) * np.float32(std))


# ----------------------------------------------------------------------------------------
# workloads
# ----------------------------------------------------------------------------------------
@dataclass(frozen=True)
class Linear:
    name: str
    d: int  # input features (contraction axis)
    n: int  # output features


@dataclass(frozen=True)
class Workload:
    name: str
    m: int
    linears: Tuple[Linear, ...]
    outlier_frac: float
    outlier_scale: float
    dist: str = "normal"
    formats: Tuple[str, ...] = ("hif4", "mxfp4")
    sparsity: Tuple[str, ...] = ("2:4",)
    backward: bool = False
    notes: str = ""


_QWEN3B = (
    Linear("qkv", 2048, 2560),
    Linear("o", 2048, 2048),
    Linear("gate_up", 2048, 22016),
    Linear("down", 11008, 2048),
)
_QWEN7B = (
    Linear("qkv", 3584, 4608),
    Linear("o", 3584, 3584),
    Linear("gate_up", 3584, 37888),
    Linear("down", 18944, 3584),
)

WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in (
        Workload("single_m16", 16, (Linear("proj", 2048, 2048),), 0.01, 50.0,
                 formats=("mxfp4", "hif4"), sparsity=("2:4",)),
        Workload("qwen3b_layer_m256", 256, _QWEN3B, 0.01, 50.0,
                 formats=("hif4", "mxfp4"), sparsity=("2:4",)),
        Workload("qwen7b_layer_m512", 512, _QWEN7B, 0.005, 100.0,
                 formats=("hif4", "mxfp4"), sparsity=("unstructured50", "block32x64_50",
                                                      "channel50")),
        Workload("qwen7b_prefill_m8192", 8192, (_QWEN7B[3], _QWEN7B[2]), 0.005, 100.0,
                 dist="t3", formats=("hif4", "mxfp4"), sparsity=("2:4",)),
        Workload("qwen3b_gateup_bwd_m8192", 8192, (_QWEN3B[2],), 0.01, 50.0,
                 formats=("hif4", "mxfp4"), sparsity=(), backward=True),
    )
}


def workload_tensors(wl: Workload, linear: Linear, seed: int = 0, m: int | None = None,
                     n_w: int | None = None):
    """Seeded (X, W[, dY]) bf16 bit arrays for one linear of a workload.

    Every linear gets its own child streams (keyed by its position in the workload), so a
    linear's tensors do not depend on which other linears are generated.  ``m`` overrides
    the token count and ``n_w`` the number of weight rows (output features) drawn; both give
    a prefix of the full draw (used to take a bounded sample of the same tensors).
    """
    idx = [l.name for l in wl.linears].index(linear.name)
    rx, rw, rg = rng_tree(seed * 1000 + idx, 3)
    mm = wl.m if m is None else m
    x = activations(rx, mm, linear.d, wl.outlier_frac, wl.outlier_scale, wl.dist)
    w = weights(rw, linear.n if n_w is None else min(n_w, linear.n), linear.d)
    if wl.backward:
        return x, w, grad_output(rg, mm, linear.n)
    return x, w
