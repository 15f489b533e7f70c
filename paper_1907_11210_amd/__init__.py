"""MI355X-native phase-decomposed transposed and dilated convolution (HUGE^2,
arXiv 1907.11210).

The computation lives in ``libhuge2.so`` (HIP kernels for gfx950 behind the C
ABI of ``include/huge2.h``); :mod:`paper_1907_11210_amd.huge2` is its Python
binding.  :mod:`paper_1907_11210_amd.workloads` generates the seeded synthetic
inputs of the benchmark and the tests.
"""
from .huge2 import (  # noqa: F401
    Plan, conv2d_dilated, conv2d_transpose, huge2_conv2d_dilated, huge2_conv2d_transpose,
    huge2_output_shape, huge2_plan_create, huge2_plan_describe, huge2_plan_destroy,
    huge2_plan_execute, huge2_plan_macs, huge2_plan_run_gemm, huge2_plan_stage_input,
    huge2_plan_kernel, huge2_plan_stages_input, make_desc,
    conv2d_transpose_wgrad, conv2d_dilated_wgrad, conv2d_transpose_dgrad, conv2d_dilated_dgrad,
    huge2_wgrad_plan_create, huge2_wgrad_execute, huge2_wgrad_plan_destroy,
    huge2_conv2d_transpose_wgrad, huge2_conv2d_dilated_wgrad,
)
