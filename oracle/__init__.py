"""CPU oracle for the Rollout-ResQ FP4 linear layer (test infrastructure only).

This package is a plain, slow, obviously-correct NumPy statement of what the GPU path
computes.  It exists to check the GPU library: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no code with the HIP
kernels, their C ABI or their Python binding, and the product path never calls it.

Floating point work is done in float64 (every dequantized value and every product of two
dequantized values is exact in float64); results that the GPU returns in float32 are rounded
to float32 once, at the end.

Contents
--------
``formats``  E2M1 / MXFP4 (paper Sec. 3, OCP MX block scaling) and HiF4 (paper Sec. 3,
             three-level hierarchical scaling, under the reading stated in that module).
``resq``     residual (Eq. 2), the sparsity functions S (Sec. 4.3), the forward of Eq. 1,
             Eq. 3 and Eq. 4, the mixed-precision W4A16 / W16A4 linears of Table 1, the FP4
             backward GEMMs of the training policy, and the overhead cost model of Sec. 5.4.

Pins: every function here is checked by ``tests/test_oracle_*.py`` against facts fixed
outside this package (value sets, exhaustive bf16 sweeps against independent integer
implementations, brute force on tiny inputs, invariants and closed forms).  The HiF4
functions are pinned to the reading written in ``formats``; whether that reading equals the
external HiF4 specification is not checked (the specification is not available here), so
the HiF4 *format definition itself* is "parity unpinned" against that specification.
"""
from . import formats, resq  # noqa: F401
