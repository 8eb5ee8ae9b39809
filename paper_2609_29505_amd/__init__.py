"""MI355X-native scheduled denoiser step of Spectral-Guided Diffusion.

The compute path is ``lib/libsgd.so`` (HIP kernels for gfx950 behind the C ABI
declared in ``include/sgd.h``).  This package only marshals arguments: PyTorch
provides device memory and streams.  Importing the binding raises if the library
has not been built (``python -m paper_2609_29505_amd.build``); there is no CPU
fallback.
"""
from .binding import (  # noqa: F401
    SGD_ARCH, SGD_BF16, SGD_F32, SGD_K, SGD_ROLE, SgdError, lib, lib_path,
    schedule_build, matrix_stats, schedule_from_scores, schedule_from_lifetimes, schedule_from_stats,
    SGD_RULE, SGD_UNIT, Schedule, DeviceModel, Cache, Graph, s_min_default, budget_layer_steps,
    op_linear, op_linear_split, op_attention, op_norm, op_norm_fold, op_frozen_run, op_heads, op_residual,
    op_adaln_mod,
    op_group_norm_silu, op_conv3x3,
)
