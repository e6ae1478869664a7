"""Seeded synthetic inputs shared by the fp64 oracle and the HIP path.

This package only *generates data*: stage shapes, seeded random tensors,
bf16 rounding of those tensors, and the op lists (schedules) that drive a
stage.  It holds none of the stage's arithmetic, so the oracle and the GPU
path can both consume it without sharing any compute code.
"""
from .configs import StageConfig, CONFIGS, TEST_CONFIGS, get_config  # noqa: F401
from .rng import (  # noqa: F401
    round_bf16, bf16_bits, bf16_bits_to_f32, gen_param, gen_params,
    gen_x, gen_dy, wshuffle_perm, PARAM_NAMES, PARAM_SHAPES, is_matrix_param,
)
from .schedules import Op, op_list, MB  # noqa: F401
