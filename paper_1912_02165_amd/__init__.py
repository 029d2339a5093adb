"""Fused Winograd 3x3 convolution for AMD MI355X (gfx950).

The compute path is the HIP library ``libwino_conv.so`` behind the C ABI of
``include/wino_conv.h`` and ``include/wino_tune.h``; ``wino`` is its Python binding and ``workloads`` draws
the seeded synthetic layers.  Importing the package does not load the library;
the first binding call does, and fails loudly if it is not built.
"""

from .wino import (  # noqa: F401
    ALGOS, Plan, WinoError, WinoTuning, conv2d, lib,
    WINO_ALGO_FFT, WINO_ALGO_FUSED, WINO_ALGO_THREE_STAGE, WINO_BUF_INPUT, WINO_BUF_PRODUCT, WINO_BUF_WEIGHTS,
    WINO_EKERNEL, WINO_MAX_CHANNEL_SPLITS,
    wino_conv_copy_intermediate, wino_conv_debug_set_status, wino_conv_describe, wino_conv_destroy,
    wino_conv_info, wino_conv_intermediate_dims, wino_conv_plan, wino_conv_plan_ex, wino_conv_run,
    wino_conv_run_noalloc, wino_conv_run_pretransformed, wino_conv_set_weights, wino_conv_status, wino_conv_workspace_bytes,
    wino_last_error, wino_fused_blockings,
    WINO_TUNE_ALL_M, WINO_TUNE_M2, WINO_TUNE_M4, WINO_TUNE_M5, WINO_TUNE_M6, WINO_TUNE_M7, WINO_TUNE_THREE_STAGE, WINO_TUNE_FFT,
    wino_conv_plan_params, wino_conv_plan_tuned, wino_wisdom_clear, wino_wisdom_load,
    wino_wisdom_lookup, wino_wisdom_save, wino_wisdom_size,
)
