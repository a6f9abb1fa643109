"""Sparse 1x1 convolution (sparse weights x dense CHW activations) for MI355X.

The work happens in ``libspconv.so`` (C ABI in include/spconv.h): a host
planner packs CSR / 1x2 / 1x4 block-CSR weights (or converts dense masked
ones), and hand-written gfx950 HIP kernels compute act(W X + b) on NCHW fp32
or fp16 tensors, optionally with a depthwise 3x3 stage fused in front.  This package is
the thin Python binding plus the in-tree build script.
"""

from .spconv import (  # noqa: F401
    Plan,
    SpconvError,
    load_library,
    spconv_dense_to_bcsr,
    spconv_dense_to_bcsr_blocked,
    spconv_conv3x3_hwc,
    spconv_depthwise3x3,
    spconv_destroy,
    spconv_global_avg_pool,
    spconv_detect_block_rows,
    spconv_detect_blocks,
    spconv_last_error,
    spconv_linear,
    spconv_options_init,
    spconv_plan_create,
    spconv_plan_create_blocked,
    spconv_plan_create_dense,
    spconv_plan_create_dense_blocked,
    spconv_plan_create_fused,
    spconv_plan_create_static,
    SPCONV_STATIC_PLAN_BYTES,
    spconv_plan_get_info,
    spconv_plan_unpack,
    spconv_plan_unpack_interleaved,
    spconv_plan_unpack_indexed,
    spconv_plan_unpack_outer,
    spconv_plan_check,
    spconv_plan_set_wait_limit,
    SPCONV_FLAG_WAIT_GAVE_UP,
    spconv_run,
)
