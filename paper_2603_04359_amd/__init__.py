"""MI355X (gfx950) implementation of the block Concentration-Alignment
Transform (CAT) W4A4 linear-layer hot path.

The compute lives in libcat.so (HIP kernels + C++ host code behind the C ABI
of include/cat.h); this package is its thin Python binding.
"""
from .binding import *  # noqa: F401,F403
from .binding import (CatError, EXPORTED, LIB_PATH, lib,  # noqa: F401
                      cat_build_transform, cat_cov_accumulate, cat_cov_workspace_bytes,
                      cat_last_error,
                      cat_quantize_weights, cat_sqnr, cat_sqnr_workspace_bytes,
                      cat_transform_quant, cat_transform_quant_workspace_bytes,
                      cat_version, cat_w4a4_linear)
