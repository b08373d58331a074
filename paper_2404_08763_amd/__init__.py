"""CATS gated-MLP hot path for AMD Instinct MI355X (gfx950).

CATS (Contextually-Aware Thresholding for Sparsity, Lee et al., COLM 2024)
wraps the SiLU of a gated MLP in a magnitude cutoff t calibrated per block
(Eq. 3-5) and then reads only the W_up / W_down rows of the neurons that
survive (Section 4.3).  The work runs in hand-written HIP kernels inside
libcats.so behind a C ABI (include/cats.h); this package is its ctypes
binding.  Build with ``python -m paper_2404_08763_amd.build``.
"""
from ._lib import (  # noqa: F401
    CATS_BF16,
    CATS_UNFUSED_INDEX,
    CATS_UNFUSED_MASK,
    CATS_F32,
    CatsError,
    Layer,
    calib_activations,
    calibrate_threshold,
    layer_from_math,
    lib_path,
    mlp_dense,
    mlp_forward,
    mlp_forward_topk,
    mlp_forward_unfused,
    pack_weights,
    raw,
    Stack,
    calibrate_stack,
    rmsnorm,
    sparse_input_gemv,
    sparse_input_workspace,
    stack_forward,
    threshold_from_acts,
    stream_read,
    timer_enable,
    timer_read,
    timer_reset,
    version,
    workspace,
    workspace_bytes,
)
