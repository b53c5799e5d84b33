"""Rollout-ResQ FP4 linear layer for AMD Instinct MI355X (gfx950).

The computation lives in ``libresq.so`` (hand-written HIP kernels behind the C ABI of
``include/resq.h``); this package only builds it (``build``) and binds it (``resq``).
"""
from .resq import (  # noqa: F401
    EXPORTED,
    FORMATS,
    SPARSITY,
    ResqError,
    library_path,
    linear_bwd,
    linear_fwd,
    load,
    quantize,
    residual_sparsify,
    resq_last_error,
    resq_linear_bwd,
    resq_linear_fwd,
    resq_quantize,
    resq_residual_sparsify,
    resq_version,
    resq_workspace_size,
    workspace,
)
