"""MI355X (gfx950) Rotated Runtime Smooth W4A4 linear layer.

A thin ctypes binding over librrs.so, the C-ABI HIP library declared in
include/rrs.h. The binding only marshals arguments: it checks torch tensors
(device, dtype, shape, contiguity), passes their device pointers and the
current HIP stream, and raises RuntimeError on a non-zero status. Every step of
the computation runs in the library's kernels. There is no fallback: if
librrs.so is missing, every call raises.

Paper: "Rotated Runtime Smooth: Training-Free Activation Smoother for accurate
INT4 inference" (arXiv 2409.20361), Sections 3.1-3.3.
"""
from __future__ import annotations

from ._binding import (  # noqa: F401
    REORDER_BLOCK,
    SCHEME_PER_CHANNEL,
    SCHEME_RUNTIME_SMOOTH,
    SCHEME_SUB_CHANNEL,
    SKIP_ROTATION,
    SKIP_SMOOTHING,
    WEIGHT_TILED,
    RRSError,
    lib,
    lib_path,
    linear,
    linear_noalloc,
    linear_reorder,
    linear_reorder_workspace_bytes,
    linear_workspace_bytes,
    prepare_weight,
    prepare_weight_sub_channel,
    quant_rows_wait_hook,
    quant_reorder_wait_hook,
    quantize_sub_channel,
    rotate_smooth_quant,
    rotate_smooth_quant_reorder,
    reorder_workspace_bytes,
    status_string,
    version,
    w4a4_gemm,
    w4a4_gemm_partials,
    w4a4_gemm_per_channel,
    w4a4_gemm_reorder,
    w4a4_gemm_scheme,
    workspace_bytes,
)

__all__ = [
    "REORDER_BLOCK", "SCHEME_PER_CHANNEL", "SCHEME_RUNTIME_SMOOTH", "SCHEME_SUB_CHANNEL",
    "SKIP_ROTATION", "SKIP_SMOOTHING", "WEIGHT_TILED", "RRSError", "lib", "lib_path", "linear", "linear_noalloc", "linear_reorder",
    "linear_reorder_workspace_bytes", "linear_workspace_bytes",
    "prepare_weight", "prepare_weight_sub_channel", "quant_rows_wait_hook",
    "quant_reorder_wait_hook",
    "quantize_sub_channel",
    "reorder_workspace_bytes", "rotate_smooth_quant", "rotate_smooth_quant_reorder",
    "status_string", "version", "w4a4_gemm", "w4a4_gemm_partials",
    "w4a4_gemm_per_channel", "w4a4_gemm_reorder", "w4a4_gemm_scheme", "workspace_bytes",
]
