"""Python binding of one decoupled-backprop pipeline stage (see include/recycle_stage.h).

Argument marshalling only: every step of the stage runs in the HIP library.
PyTorch supplies the three device arenas and the HIP stream, nothing else.
"""
from __future__ import annotations

import ctypes
from typing import List, Optional, Sequence, Tuple

import numpy as np

from . import _lib as L

PARAM_NAMES = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
               "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2")


def param_shape(pid: int, hidden: int, ffn: int) -> Tuple[int, ...]:
    h, f = hidden, ffn
    return ((h,), (h,), (h, 3 * h), (3 * h,), (h, h), (h,),
            (h,), (h,), (h, f), (f,), (f, h), (h,))[pid]


def _mb(mb) -> L.RcMb:
    if isinstance(mb, L.RcMb):
        return mb
    if isinstance(mb, int):
        return L.RcMb(mb, 0)
    return L.RcMb(int(mb[0]), int(mb[1]) if len(mb) > 1 else 0)


class Stage:
    """Stage i = ``stage_index`` of data-parallel pipeline k_s = ``pipeline_id``.

    ``dry_run=True`` creates a bookkeeping-only handle (no device memory, no
    kernels): it validates op lists on the host.  ``static_work=True`` creates
    the handle with rc_stage_create_static: its work memory is the library's
    own per-device array, so only the state and stash arenas are allocated
    here."""

    def __init__(self, *, num_layers: int, hidden: int, heads: int, ffn: int, seq_len: int,
                 micro_batch: int, causal: bool = True, dtype: str = "bf16",
                 ln_eps: float = 1e-5, max_stashed_mb: int = 1, max_inflight_mb: Optional[int] = None,
                 lr: float = 1e-4, beta1: float = 0.9, beta2: float = 0.95, eps: float = 1e-8,
                 weight_decay: float = 0.1, stage_index: int = 0, pipeline_id: int = 0,
                 device=None, stream=None, dry_run: bool = False, static_work: bool = False):
        self._lib = L.load()
        self._h = None
        if dtype not in ("bf16", "f32"):
            raise ValueError("dtype must be 'bf16' or 'f32'")
        self.dtype = dtype
        self.cfg = L.RcStageConfig(num_layers, hidden, heads, ffn, seq_len, micro_batch,
                                   1 if causal else 0, L.RC_BF16 if dtype == "bf16" else L.RC_FP32,
                                   ln_eps, max_stashed_mb,
                                   max_inflight_mb if max_inflight_mb is not None else max_stashed_mb)
        self.adam = L.RcAdamConfig(lr, beta1, beta2, eps, weight_decay)
        st, sh, wk = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
        L.check(self._lib.rc_stage_memory_requirements(ctypes.byref(self.cfg), ctypes.byref(st),
                                                       ctypes.byref(sh), ctypes.byref(wk)))
        self.state_bytes, self.stash_bytes, self.work_bytes = st.value, sh.value, wk.value
        self.dry_run = dry_run
        handle = ctypes.c_void_p()
        if dry_run:
            L.check(self._lib.rc_stage_create(ctypes.byref(self.cfg), ctypes.byref(self.adam),
                                              stage_index, pipeline_id, None, None, None, None,
                                              ctypes.byref(handle)))
        else:
            import torch
            if not torch.cuda.is_available():
                raise RuntimeError("no HIP device: the stage runs only on the GPU")
            self.device = torch.device(device if device is not None else "cuda")
            sizes = (self.state_bytes, self.stash_bytes) + (() if static_work else (self.work_bytes,))
            self._arenas = [torch.empty(max(n, 256), dtype=torch.uint8, device=self.device)
                            for n in sizes]
            self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
            create = self._lib.rc_stage_create_static if static_work else self._lib.rc_stage_create
            L.check(create(
                ctypes.byref(self.cfg), ctypes.byref(self.adam), stage_index, pipeline_id,
                *[ctypes.c_void_p(a.data_ptr()) for a in self._arenas],
                ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(handle)))
        self._h = handle

    @classmethod
    def from_config(cls, cfg, **kw) -> "Stage":
        """Build from any object with the workload attributes (layers, hidden,
        heads, ffn, seq, micro_batch, causal, dtype, ln_eps, stash_slots,
        inflight_slots)."""
        return cls(num_layers=cfg.layers, hidden=cfg.hidden, heads=cfg.heads, ffn=cfg.ffn,
                   seq_len=cfg.seq, micro_batch=cfg.micro_batch, causal=cfg.causal,
                   dtype=cfg.dtype, ln_eps=cfg.ln_eps,
                   max_stashed_mb=kw.pop("max_stashed_mb", cfg.stash_slots),
                   max_inflight_mb=kw.pop("max_inflight_mb", cfg.inflight_slots), **kw)

    # -- lifetime -------------------------------------------------------------
    def close(self) -> None:
        if self._h is not None and self._h.value:
            h, self._h = self._h, None
            L.check(self._lib.rc_stage_destroy(h))

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- helpers --------------------------------------------------------------
    @property
    def act_shape(self):
        return (self.cfg.micro_batch, self.cfg.seq_len, self.cfg.hidden)

    def _torch_dtype(self):
        import torch
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def _check_act(self, t, name):
        import torch
        if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
            raise TypeError(f"{name} must be a device tensor")
        if t.dtype != self._torch_dtype() or tuple(t.shape) != self.act_shape or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {self.act_shape} {self.dtype} tensor")
        return ctypes.c_void_p(t.data_ptr())

    def _new_act(self):
        import torch
        return torch.empty(self.act_shape, dtype=self._torch_dtype(), device=self.device)

    # -- the four calls of the stage ---------------------------------------------
    def forward(self, mb, x=None, y=None):
        """F of micro-batch (j, k): y = Stage(x)."""
        if self.dry_run:
            L.check(self._lib.rc_stage_forward(self._h, _mb(mb), None, None))
            return None
        y = self._new_act() if y is None else y
        L.check(self._lib.rc_stage_forward(self._h, _mb(mb), self._check_act(x, "x"),
                                           self._check_act(y, "y")))
        return y

    def backward_input(self, mb, dy=None, dx=None):
        """B_input of micro-batch (j, k): dx = J_x^T dy; no parameter gradient."""
        if self.dry_run:
            L.check(self._lib.rc_stage_backward_input(self._h, _mb(mb), None, None))
            return None
        dx = self._new_act() if dx is None else dx
        L.check(self._lib.rc_stage_backward_input(self._h, _mb(mb), self._check_act(dy, "dy"),
                                                  self._check_act(dx, "dx")))
        return dx

    def backward(self, mb, dy=None, dx=None):
        """Coupled backward of micro-batch (j, k): B_input then its B_weight."""
        if self.dry_run:
            L.check(self._lib.rc_stage_backward(self._h, _mb(mb), None, None))
            return None
        dx = self._new_act() if dx is None else dx
        L.check(self._lib.rc_stage_backward(self._h, _mb(mb), self._check_act(dy, "dy"),
                                            self._check_act(dx, "dx")))
        return dx

    def stash_account(self, reset_peak: bool = False) -> dict:
        """Stash bytes: a_f, s_w per micro-batch; live, peak, limit."""
        a = L.RcStashAccount()
        L.check(self._lib.rc_stage_stash_account(self._h, ctypes.byref(a), int(bool(reset_peak))))
        return {"a_f": a.a_f, "s_w": a.s_w, "live": a.live, "peak": a.peak, "limit": a.limit}

    def set_stash_limit(self, nbytes: int) -> None:
        """Stash limit (bytes, 0 = none) that forward passes respect."""
        L.check(self._lib.rc_stage_set_stash_limit(self._h, ctypes.c_uint64(int(nbytes))))

    def backward_weight(self, mb) -> None:
        """B_weight of micro-batch (j, k): accumulate its parameter gradients."""
        L.check(self._lib.rc_stage_backward_weight(self._h, _mb(mb)))

    def backward_weight_many(self, mbs) -> None:
        """B_weight of several micro-batches in one pass (same result as one
        call per micro-batch in this order; one product per parameter over
        their concatenated tokens)."""
        mbs = list(mbs)
        arr = (L.RcMb * max(1, len(mbs)))(*[_mb(m) for m in mbs])
        L.check(self._lib.rc_stage_backward_weight_many(self._h, arr, len(mbs)))

    def optimizer_step(self, grad_scale: float = 1.0) -> None:
        """This stage's AdamW step (no cross-stage synchronisation)."""
        L.check(self._lib.rc_stage_optimizer_step(self._h, float(grad_scale)))

    def grad_check(self, grad_scale: float = 1.0):
        """Post-step local validation: (sum of squares, non-finite count) of
        grad_scale * the gradient."""
        ss, bad = ctypes.c_double(), ctypes.c_int64()
        L.check(self._lib.rc_stage_grad_check(self._h, float(grad_scale), ctypes.byref(ss),
                                              ctypes.byref(bad)))
        return ss.value, bad.value

    def optimizer_skip(self) -> None:
        """Close the iteration without an update."""
        L.check(self._lib.rc_stage_optimizer_skip(self._h))

    def optimizer_rollback(self) -> None:
        """Undo the optimizer step that was the last call."""
        L.check(self._lib.rc_stage_optimizer_rollback(self._h))

    # -- state access -----------------------------------------------------------
    def load_param(self, layer: int, pid: int, value) -> None:
        a = np.ascontiguousarray(value, dtype=np.float32)
        if a.shape != param_shape(pid, self.cfg.hidden, self.cfg.ffn):
            raise ValueError(f"param {PARAM_NAMES[pid]} has shape "
                             f"{param_shape(pid, self.cfg.hidden, self.cfg.ffn)}, got {a.shape}")
        L.check(self._lib.rc_stage_load_param(self._h, layer, pid, a.ctypes.data_as(ctypes.c_void_p)))

    def load_params(self, params: Sequence[Sequence[np.ndarray]]) -> None:
        for l, layer in enumerate(params):
            for pid, v in enumerate(layer):
                self.load_param(l, pid, v)

    def read(self, what: int, layer: int, pid: int) -> np.ndarray:
        out = np.empty(param_shape(pid, self.cfg.hidden, self.cfg.ffn), dtype=np.float32)
        L.check(self._lib.rc_stage_read(self._h, what, layer, pid, out.ctypes.data_as(ctypes.c_void_p)))
        return out

    def read_all(self, what: int) -> List[List[np.ndarray]]:
        return [[self.read(what, l, p) for p in range(L.RC_NUM_PARAMS)]
                for l in range(self.cfg.num_layers)]

    def op_log(self) -> List[Tuple[int, int, int, int, int, int]]:
        """Records (seq, op, j, k, k_s, iter) in issue order."""
        n = ctypes.c_int32()
        L.check(self._lib.rc_stage_op_log(self._h, None, 0, ctypes.byref(n)))
        buf = (L.RcOpRecord * max(n.value, 1))()
        L.check(self._lib.rc_stage_op_log(self._h, buf, n.value, ctypes.byref(n)))
        return [(r.seq, r.op, r.j, r.k, r.k_s, r.iter) for r in buf[:n.value]]

    def stash_usage(self) -> Tuple[int, int]:
        a, b = ctypes.c_int32(), ctypes.c_int32()
        L.check(self._lib.rc_stage_stash_usage(self._h, ctypes.byref(a), ctypes.byref(b)))
        return a.value, b.value

    def attention_kernels(self) -> str:
        """Which attention kernels F and B_input run: "materialised", "block"
        or "paired" (chosen from the shape and the device's compute units)."""
        k = ctypes.c_int32()
        L.check(self._lib.rc_stage_attention_kernels(self._h, ctypes.byref(k)))
        return {L.RC_ATTN_MATERIALISED: "materialised", L.RC_ATTN_BLOCK: "block",
                L.RC_ATTN_PAIRED: "paired"}[k.value]

    def set_stream(self, stream) -> None:
        self.stream = stream
        L.check(self._lib.rc_stage_set_stream(self._h, ctypes.c_void_p(stream.cuda_stream)))

    def profile_enable(self, enable: bool = True) -> None:
        """Start (resetting the counters) or stop the per-kernel-class profile."""
        L.check(self._lib.rc_stage_profile_enable(self._h, 1 if enable else 0))

    def profile_read(self) -> dict:
        """{class: {launches, ms, flops, bytes}} accumulated since profile_enable()."""
        buf = (L.RcKernelStat * len(L.KERNEL_CLASSES))()
        L.check(self._lib.rc_stage_profile_read(self._h, buf))
        return {L.KERNEL_CLASSES[r.kind]: dict(launches=r.launches, ms=r.ms, flops=r.flops,
                                               bytes=r.bytes) for r in buf}

    def synchronize(self) -> None:
        L.check(self._lib.rc_stage_synchronize(self._h))
