"""MI355X-native action-guided sparse denoising step (Sparse-WAM hot path).

The compute lives in libswam.so (hand-written HIP for gfx950, C ABI in
include/swam.h); this package is its thin Python binding.
"""
from .swam import (  # noqa: F401
    Config, Context, Model, PlanInfo, SwamError, load_library, plan, LIB_PATH, EXPORTS,
    FORCE_DENSE, FORCE_REFRESH, KIND_DENSE, KIND_REFRESH, KIND_SPARSE, TIMERS, WEIGHT_NAMES,
    SWAM_F32, SWAM_BF16,
)
