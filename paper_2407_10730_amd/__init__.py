"""MI355X (gfx950) conv2d forward primitive with a ConvBench-style phase breakdown.

The library (libconv2d.so, HIP) exports the C ABI declared in
include/conv2d.h; ``binding`` mirrors it function by function and
``runner`` drives one operation with torch-owned device memory.
"""
from .binding import (  # noqa: F401
    ALGO_NAMES, CONV2D_ALGO_AUTO, CONV2D_ALGO_DIRECT, CONV2D_ALGO_IM2COL_GEMM,
    CONV2D_ALGO_IMPLICIT_GEMM, CONV2D_BF16, CONV2D_F32, CONV2D_NCHW, CONV2D_NHWC, PHASE_NAMES,
    Conv2dError, conv2d_breakdown, conv2d_breakdown_reset, conv2d_desc_create,
    conv2d_desc_destroy, conv2d_fwd, conv2d_output_shape, conv2d_params, conv2d_plan_query,
    conv2d_runtime_version, conv2d_set_timing, conv2d_status_string, load)
