"""Parameterized fp32 GEMM and NHWC convolution forward for AMD MI355X (gfx950).

The compute path is libpk.so (hand-written HIP kernels behind the C-ABI in
include/pk.h); this package only marshals arguments into it.
"""
from .binding import (PkError, PkLibraryMissing, configs, conv2d_fwd, conv2d_out_dims,  # noqa: F401
                      conv2d_same_pads, conv2d_winograd, conv2d_winograd_workspace_bytes,
                      conv2d_workspace_bytes, force_config, force_splits, gemm, tune_conv2d, tune_gemm,
                      tune_reset,
                      last_config_name, last_invalid_param, load)
