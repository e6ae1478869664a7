"""Schedule-side calls of the library (host only): Failure Normalization
(section 4.2.1, Algorithm 1) and the unit-slot schedule simulator (sections
3.1-3.3), whose per-worker op lists drive a stage handle through
``executor.execute``."""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Dict, List, Sequence, Tuple

from . import _lib as L

RC_SIM_MAX_ITER = 16


class RcSimConfig(ctypes.Structure):
    _fields_ = [("dp", ctypes.c_int32), ("pp", ctypes.c_int32), ("mb", ctypes.c_int32),
                ("decoupled", ctypes.c_int32), ("staggered", ctypes.c_int32),
                ("iterations", ctypes.c_int32), ("inflight_cap", ctypes.c_int32),
                ("n_failed", ctypes.c_int32), ("failed", ctypes.POINTER(ctypes.c_int32))]


class RcSimResult(ctypes.Structure):
    _fields_ = [("makespan", ctypes.c_int32), ("workers", ctypes.c_int32), ("busy_max", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("iter_end", ctypes.c_int32 * RC_SIM_MAX_ITER)]


class RcSimOp(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("slot", "op", "iter", "stage", "j", "k", "k_s", "dur")]


def failure_normalization(dp: int, pp: int, mb: int, failures: int) -> Tuple[List[int], int]:
    """(failures per stage, estimated extra slots)."""
    lib = L.load()
    per = (ctypes.c_int32 * max(1, pp))()
    ov = ctypes.c_int64()
    L.check(lib.rc_failure_normalization(dp, pp, mb, failures, per, ctypes.byref(ov)))
    return list(per)[:pp], ov.value


@dataclass
class SimOp:
    slot: int
    kind: str        # "F" | "B" | "W"
    iteration: int
    stage: int
    j: int
    k: int           # origin pipeline
    k_s: int         # executing pipeline
    dur: int


@dataclass
class SimResult:
    makespan: int
    iter_end: List[int]
    busy_max: int
    ops: List[SimOp]

    def worker_ops(self, k_s: int, stage: int) -> List[SimOp]:
        """The op list of worker (k_s, stage) in start order."""
        return [o for o in self.ops if o.k_s == k_s and o.stage == stage]


def simulate(dp: int, pp: int, mb: int, failed: Sequence[Tuple[int, int]] = (), decoupled: bool = False,
             staggered: bool = False, iterations: int = 1, inflight_cap: bool = False) -> SimResult:
    lib = L.load()
    fl = (ctypes.c_int32 * max(1, 2 * len(failed)))(*[v for kv in failed for v in kv])
    cfg = RcSimConfig(dp, pp, mb, int(decoupled), int(staggered), iterations, int(inflight_cap),
                      len(failed), fl)
    res = RcSimResult()
    n = ctypes.c_int32()
    L.check(lib.rc_schedule_simulate(ctypes.byref(cfg), ctypes.byref(res), None, 0, ctypes.byref(n)))
    buf = (RcSimOp * max(1, n.value))()
    L.check(lib.rc_schedule_simulate(ctypes.byref(cfg), ctypes.byref(res), buf, n.value, ctypes.byref(n)))
    kinds = {L.RC_OP_F: "F", L.RC_OP_B: "B", L.RC_OP_W: "W"}
    ops = [SimOp(o.slot, kinds[o.op], o.iter, o.stage, o.j, o.k, o.k_s, o.dur) for o in buf[:n.value]]
    return SimResult(res.makespan, list(res.iter_end)[:iterations], res.busy_max, ops)
