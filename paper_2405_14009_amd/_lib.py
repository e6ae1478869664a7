"""ctypes declarations of the C ABI in include/recycle_stage.h.

Loading fails loudly when the HIP library has not been built: there is no
fallback implementation of any call.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librecycle_stage.so")

RC_OK, RC_ERR_INVALID_ARG, RC_ERR_BAD_STATE, RC_ERR_OUT_OF_STASH, RC_ERR_HIP, RC_ERR_UNSUPPORTED = (
    0, -1, -2, -3, -4, -5)
RC_FP32, RC_BF16 = 0, 1
RC_OP_F, RC_OP_B, RC_OP_W, RC_OP_STEP, RC_OP_SKIP, RC_OP_ROLLBACK = 0, 1, 2, 3, 4, 5
RC_READ_PARAM, RC_READ_GRAD, RC_READ_ADAM_M, RC_READ_ADAM_V = 0, 1, 2, 3
RC_NUM_PARAMS = 12
RC_ATTN_MATERIALISED, RC_ATTN_BLOCK, RC_ATTN_PAIRED = 0, 1, 2
RC_STATIC_WORK_BYTES = 96 * 1024 * 1024

# Every symbol the header declares, for load checks.
EXPORTED = (
    "rc_stage_memory_requirements", "rc_stage_create", "rc_stage_create_static", "rc_stage_destroy", "rc_stage_load_param",
    "rc_stage_read", "rc_stage_forward", "rc_stage_backward_input", "rc_stage_backward",
    "rc_stage_backward_weight", "rc_stage_stash_account", "rc_stage_set_stash_limit",
    "rc_stage_backward_weight_many", "rc_stage_optimizer_step", "rc_stage_grad_check",
    "rc_stage_optimizer_skip", "rc_stage_optimizer_rollback", "rc_stage_op_log",
    "rc_stage_stash_usage", "rc_stage_set_stream", "rc_stage_attention_kernels",
    "rc_stage_synchronize", "rc_stage_profile_enable", "rc_stage_profile_read", "rc_last_error",
    "rc_failure_normalization", "rc_schedule_simulate",
)

KERNEL_CLASSES = ("gemm_fwd", "gemm_dgrad", "gemm_wgrad", "attn_fwd", "attn_bwd", "layernorm",
                  "reduce", "adamw", "copy")


class RcStashAccount(ctypes.Structure):
    _fields_ = [("a_f", ctypes.c_uint64), ("s_w", ctypes.c_uint64), ("live", ctypes.c_uint64),
                ("peak", ctypes.c_uint64), ("limit", ctypes.c_uint64)]


class RcStageConfig(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("heads", ctypes.c_int32), ("ffn", ctypes.c_int32), ("seq_len", ctypes.c_int32),
                ("micro_batch", ctypes.c_int32), ("causal", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("ln_eps", ctypes.c_float),
                ("max_stashed_mb", ctypes.c_int32), ("max_inflight_mb", ctypes.c_int32)]


class RcAdamConfig(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float)]


class RcMb(ctypes.Structure):
    _fields_ = [("j", ctypes.c_int32), ("k", ctypes.c_int32)]


class RcOpRecord(ctypes.Structure):
    _fields_ = [("seq", ctypes.c_int64), ("op", ctypes.c_int32), ("j", ctypes.c_int32),
                ("k", ctypes.c_int32), ("k_s", ctypes.c_int32), ("stage", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("iter", ctypes.c_int64)]


class RcKernelStat(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("launches", ctypes.c_int32), ("ms", ctypes.c_double),
                ("flops", ctypes.c_double), ("bytes", ctypes.c_double)]


class RcError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"[{_NAMES.get(status, status)}] {msg}")
        self.status = status


class InvalidArgError(RcError): pass
class BadStateError(RcError): pass
class OutOfStashError(RcError): pass
class HipError(RcError): pass
class UnsupportedError(RcError): pass


_NAMES = {RC_ERR_INVALID_ARG: "RC_ERR_INVALID_ARG", RC_ERR_BAD_STATE: "RC_ERR_BAD_STATE",
          RC_ERR_OUT_OF_STASH: "RC_ERR_OUT_OF_STASH", RC_ERR_HIP: "RC_ERR_HIP",
          RC_ERR_UNSUPPORTED: "RC_ERR_UNSUPPORTED"}
_EXC = {RC_ERR_INVALID_ARG: InvalidArgError, RC_ERR_BAD_STATE: BadStateError,
        RC_ERR_OUT_OF_STASH: OutOfStashError, RC_ERR_HIP: HipError,
        RC_ERR_UNSUPPORTED: UnsupportedError}

_lib = None


def load() -> ctypes.CDLL:
    """The HIP library, loaded once.  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2405_14009_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, F32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
    cfgp = ctypes.POINTER(RcStageConfig)
    sz = ctypes.POINTER(ctypes.c_size_t)
    sig = {
        "rc_stage_memory_requirements": [cfgp, sz, sz, sz],
        "rc_stage_create": [cfgp, ctypes.POINTER(RcAdamConfig), I32, I32, P, P, P, P,
                            ctypes.POINTER(P)],
        "rc_stage_create_static": [cfgp, ctypes.POINTER(RcAdamConfig), I32, I32, P, P, P,
                                   ctypes.POINTER(P)],
        "rc_stage_destroy": [P],
        "rc_stage_load_param": [P, I32, I32, P],
        "rc_stage_read": [P, I32, I32, I32, P],
        "rc_stage_forward": [P, RcMb, P, P],
        "rc_stage_backward_input": [P, RcMb, P, P],
        "rc_stage_backward": [P, RcMb, P, P],
        "rc_stage_stash_account": [P, ctypes.POINTER(RcStashAccount), I32],
        "rc_stage_set_stash_limit": [P, ctypes.c_uint64],
        "rc_stage_backward_weight": [P, RcMb],
        "rc_stage_backward_weight_many": [P, ctypes.POINTER(RcMb), I32],
        "rc_stage_optimizer_step": [P, F32],
        "rc_stage_grad_check": [P, F32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)],
        "rc_stage_optimizer_skip": [P],
        "rc_stage_optimizer_rollback": [P],
        "rc_stage_op_log": [P, ctypes.POINTER(RcOpRecord), I32, ctypes.POINTER(I32)],
        "rc_stage_stash_usage": [P, ctypes.POINTER(I32), ctypes.POINTER(I32)],
        "rc_stage_set_stream": [P, P],
        "rc_stage_attention_kernels": [P, ctypes.POINTER(I32)],
        "rc_stage_synchronize": [P],
        "rc_stage_profile_enable": [P, I32],
        "rc_stage_profile_read": [P, ctypes.POINTER(RcKernelStat)],
        "rc_failure_normalization": [I32, I32, I32, I32, ctypes.POINTER(I32), ctypes.POINTER(ctypes.c_int64)],
        "rc_schedule_simulate": [P, P, P, I32, ctypes.POINTER(I32)],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.rc_last_error.argtypes = []
    lib.rc_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def check(status: int) -> None:
    if status != RC_OK:
        msg = load().rc_last_error().decode(errors="replace")
        raise _EXC.get(status, RcError)(status, msg)
