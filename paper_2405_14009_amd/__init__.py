"""MI355X-native decoupled-backprop pipeline stage (ReCycle, SOSP'24).

The compute lives in ``librecycle_stage.so`` (hand-written HIP for gfx950)
behind the C ABI of ``include/recycle_stage.h``; this package is its thin
Python binding.
"""
from ._lib import (  # noqa: F401
    BadStateError, HipError, InvalidArgError, OutOfStashError, RcError, UnsupportedError,
    RC_OP_B, RC_OP_F, RC_OP_ROLLBACK, RC_OP_SKIP, RC_OP_STEP, RC_OP_W, RC_READ_ADAM_M,
    RC_READ_ADAM_V, RC_READ_GRAD,
    RC_READ_PARAM, LIB_PATH, load,
)
from .stage import PARAM_NAMES, Stage, param_shape  # noqa: F401
