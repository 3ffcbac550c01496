"""QuantEase (arXiv 2309.01885) hot path for AMD MI355X (gfx950).

The computation lives in libqe.so (hand-written HIP kernels behind the C ABI
of include/qe.h); ``paper_2309_01885_amd.qe`` is its ctypes binding.
"""
from .qe import (QE_CD_DENSE, QE_CD_FP32, QE_CODES_VALID, QE_GRAM_BF16X3, QE_GRAM_FP32, QE_INIT_FROM_W, QE_LAYOUT_NP, QE_LAYOUT_PN,  # noqa: F401
                 QE_R_VALID, QE_OK, QE_ERR_ARG, QE_ERR_DIAG, QE_ERR_SCALE, QE_ERR_WORKSPACE, QE_ERR_HIP,
                 QE_ERR_UNSUPPORTED, QE_ERR_TOO_LARGE, QE_ERR_NONFINITE, QE_DEBUG_CHECKS,
                 QE_NOALLOC_SCRATCH_BYTES, QE_OBJ_IN,
                 QE_OUTLIER_COLUMNS, QE_RELAX_MASK, QE_RELAX_PERIOD,
                 QEError, cd_outlier_sweep, cd_sweep, cd_sweep_noalloc, cd_workspace_size, gram, grid_minmax,
                 lambda_max, load, objective, outliers_csr, outlier_workspace_size, pack_codes,
                 sync_status, topk_abs, topk_columns, workspace)
