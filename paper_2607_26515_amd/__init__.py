"""Rollout-ResQ FP4 linear layer for AMD Instinct MI355X (gfx950).

The computation lives in ``libresq.so`` (hand-written HIP kernels behind the C ABI of
``include/resq.h``); this package only builds it (``build``) and binds it (``resq``).
"""
from .resq import (  # noqa: F401
    EXPORTED,
    FORMATS,
    OP_LINEAR_BWD,
    OP_LINEAR_FWD,
    OP_LINEAR_FWD_PREPARED,
    OP_RESIDUAL_SPARSIFY,
    SPARSITY,
    ResqError,
    library_path,
    linear_bwd,
    linear_fwd,
    linear_fwd_prepared,
    prepare_weights,
    load,
    quantize,
    residual_sparsify,
    resq_last_error,
    resq_linear_bwd,
    resq_linear_fwd,
    resq_linear_fwd_prepared,
    resq_linear_fwd_prepared_bf16,
    resq_prepare_weights,
    resq_prepared_weights_size,
    resq_profile_enable,
    resq_profile_read,
    resq_profile_reset,
    resq_quantize,
    resq_residual_sparsify,
    resq_version,
    resq_workspace_size,
    workspace,
)
