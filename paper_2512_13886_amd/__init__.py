"""OPTIMA weight-update hot path on AMD MI355X (gfx950).

The compute lives in liboptima.so (hand-written HIP kernels behind a C ABI,
declared in include/optima.h). This package is its thin Python binding; the
names match the C entry points. Importing it fails loudly if the library has
not been built (python paper_2512_13886_amd/build.py) or is stale.
"""
from ._lib import (OptimaError, SolverOpts, DTYPE_F32, DTYPE_BF16, DTYPE_F64, PREC_FP32,
                   PREC_BF16X3, SPECTRAL_MAX_BLOCK, MASK_UNSTRUCTURED, MASK_2TO4, METHOD_RAPDHG,
                   METHOD_CG, library_path,
                   optima_status_string, optima_abi_version,
                   optima_hessian_workspace_bytes, optima_hessian_accumulate,
                   optima_hessian_damp, optima_hessian_jacobi,
                   optima_spectral_norm_workspace_bytes,
                   optima_spectral_norm, LANCZOS_MAX_STEPS,
                   SPECTRAL_NOALLOC_MAX_DIM, optima_spectral_norm_noalloc,
                   optima_spectral_lanczos_workspace_bytes, optima_spectral_lanczos,
                   optima_wanda_mask, optima_qp_workspace_bytes,
                   optima_qp_solve_batched, ACT_NONE, ACT_SILU,
                   optima_linear_forward_workspace_bytes, optima_linear_forward)

__all__ = [
    "OptimaError", "SolverOpts", "DTYPE_F32", "DTYPE_BF16", "DTYPE_F64", "PREC_FP32",
    "PREC_BF16X3", "SPECTRAL_MAX_BLOCK", "MASK_UNSTRUCTURED", "MASK_2TO4", "METHOD_RAPDHG",
    "METHOD_CG", "library_path",
    "optima_status_string", "optima_abi_version", "optima_hessian_workspace_bytes",
    "optima_hessian_accumulate", "optima_hessian_damp", "optima_hessian_jacobi",
    "optima_spectral_norm_workspace_bytes", "optima_spectral_norm", "LANCZOS_MAX_STEPS",
    "SPECTRAL_NOALLOC_MAX_DIM", "optima_spectral_norm_noalloc",
    "optima_spectral_lanczos_workspace_bytes", "optima_spectral_lanczos", "optima_wanda_mask",
    "optima_qp_workspace_bytes", "optima_qp_solve_batched", "ACT_NONE", "ACT_SILU",
    "optima_linear_forward_workspace_bytes", "optima_linear_forward",
]
