"""Schedule executor for one stage handle (host side; the compute is in the
library).

Runs an op list of the stage's worker - F, B (B_input), W (B_weight), STEP,
SKIP, ROLLBACK records for micro-batches (j, k) - through the C ABI, with
Decoupled BackProp applied selectively under a stash limit (section 3.2,
"the memory challenge"; the memory constraint of the schedule MILP, section
4.2.2):

* B of a micro-batch whose deferred weight-pass stash would raise the stash
  above the limit runs coupled (B_input and B_weight in one call); its later
  W record is then already done.
* F that would not fit first runs deferred weight passes, oldest first,
  until it does (OutOfStashError if nothing is left to run).
* Consecutive W records are run as one batched weight pass (up to 32).

The stash figures are the library's own accounting (rc_stage_stash_account).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Optional

from . import _lib as L


@dataclass
class ExecReport:
    coupled: List[tuple] = field(default_factory=list)   # micro-batches run with a coupled backward
    flushed: List[tuple] = field(default_factory=list)   # weight passes run early to admit a forward
    peak: int = 0                                         # stash peak (bytes, between calls)
    weight_calls: int = 0                                 # weight-pass library calls


def _key(mb):
    return (int(mb[0]), int(mb[1]))


def execute(stage, ops, x_fn: Optional[Callable] = None, dy_fn: Optional[Callable] = None,
            stash_limit: int = 0, batch_weights: bool = True,
            on_output: Optional[Callable] = None) -> ExecReport:
    """Run ``ops`` (objects with ``kind`` in F/B/W/STEP/SKIP/ROLLBACK and
    ``mb``) on ``stage``.  ``x_fn(mb)`` / ``dy_fn(mb)`` give device inputs
    (ignored on dry-run handles); ``on_output(kind, mb, tensor)`` receives y
    and dx."""
    rep = ExecReport()
    stage.set_stash_limit(stash_limit)
    stage.stash_account(reset_peak=True)
    deferred: List[tuple] = []      # B done, W not yet, in B order
    done_w = set()
    dry = stage.dry_run
    pending_w: List[tuple] = []

    def flush_pending():
        nonlocal pending_w
        if not pending_w:
            return
        for i in range(0, len(pending_w), 32):
            chunk = pending_w[i:i + 32]
            if len(chunk) == 1:
                stage.backward_weight(chunk[0])
            else:
                stage.backward_weight_many(chunk)
            rep.weight_calls += 1
        for mb in pending_w:
            deferred.remove(mb)
            done_w.add(mb)
        pending_w = []

    for op in ops:
        kind = op.kind
        if kind != "W":
            flush_pending()
        if kind == "F":
            mb = _key(op.mb)
            acct = stage.stash_account()
            if stash_limit:
                while acct["live"] + acct["a_f"] > stash_limit and deferred:
                    early = deferred[0]
                    stage.backward_weight(early)
                    rep.weight_calls += 1
                    deferred.remove(early)
                    done_w.add(early)
                    rep.flushed.append(early)
                    acct = stage.stash_account()
            y = stage.forward(mb, None if dry else x_fn(mb))
            if on_output and y is not None:
                on_output("F", mb, y)
        elif kind == "B":
            mb = _key(op.mb)
            acct = stage.stash_account()
            dy = None if dry else dy_fn(mb)
            if stash_limit and acct["live"] + acct["s_w"] - acct["a_f"] > stash_limit:
                dx = stage.backward(mb, dy)
                done_w.add(mb)
                rep.coupled.append(mb)
                rep.weight_calls += 1
            else:
                dx = stage.backward_input(mb, dy)
                deferred.append(mb)
            if on_output and dx is not None:
                on_output("B", mb, dx)
        elif kind == "W":
            mb = _key(op.mb)
            if mb in done_w:
                continue
            if batch_weights:
                pending_w.append(mb)
            else:
                stage.backward_weight(mb)
                rep.weight_calls += 1
                deferred.remove(mb)
                done_w.add(mb)
        elif kind == "STEP":
            if deferred:
                raise L.BadStateError(f"optimizer step with weight passes pending: {deferred}")
            stage.optimizer_step()
            done_w.clear()
        elif kind == "SKIP":
            stage.optimizer_skip()
            done_w.clear()
        elif kind == "ROLLBACK":
            stage.optimizer_rollback()
        else:
            raise ValueError(f"unknown op kind {kind!r}")
    flush_pending()
    rep.peak = stage.stash_account()["peak"]
    return rep
