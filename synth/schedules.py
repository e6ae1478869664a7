"""Op lists that drive one stage through a training iteration.

An op is (kind, micro-batch) with kind in F, B (input-gradient pass), W
(deferred weight-gradient pass) and STEP (this stage's optimizer step).  The
families follow the 1F1B schedule with decoupled backward of the paper
(Decoupled BackProp section; fault-free schedule figure): warm-up forwards,
then alternating B/F, then the remaining B, with W deferred.
"""
from __future__ import annotations

from typing import List, NamedTuple, Optional

from .rng import wshuffle_perm


class MB(NamedTuple):
    j: int      # micro-batch id within the iteration
    k: int = 0  # original data-parallel pipeline (differs from the stage's own when re-routed)


class Op(NamedTuple):
    kind: str            # "F" | "B" | "W" | "STEP"
    mb: Optional[MB] = None


def micro_batches(cfg) -> List[MB]:
    return [MB(j, cfg.reroute_origin if j in cfg.rerouted else 0) for j in range(cfg.n_mb)]


def _one_f_one_b(mbs, warmup):
    ops = [Op("F", m) for m in mbs[:warmup]]
    for i, m in enumerate(mbs[warmup:]):
        ops.append(Op("B", mbs[i]))
        ops.append(Op("F", m))
    for m in mbs[len(mbs) - warmup:] if warmup <= len(mbs) else mbs:
        ops.append(Op("B", m))
    return ops


def op_list(cfg, with_step: bool = True) -> List[Op]:
    mbs = micro_batches(cfg)
    warm = min(cfg.warmup, len(mbs))
    kind = cfg.schedule
    if kind == "tiny":
        # F0 F1 B0 F2 B1 F3 B2 B3 . W0 W1 W2 W3
        ops = _one_f_one_b(mbs, warm) + [Op("W", m) for m in mbs]
    elif kind == "1f1b_cooldown_w":
        # W passes fill the cool-down: each remaining B is followed by the
        # oldest pending W, then the rest of the W in j order.
        ops = [Op("F", m) for m in mbs[:warm]]
        for i, m in enumerate(mbs[warm:]):
            ops += [Op("B", mbs[i]), Op("F", m)]
        pend = list(mbs)
        for m in mbs[len(mbs) - warm:]:
            ops.append(Op("B", m))
            ops.append(Op("W", pend.pop(0)))
        ops += [Op("W", m) for m in pend]
    elif kind == "1f1b_deferred_shuffled_w":
        perm = wshuffle_perm(cfg, len(mbs))
        ops = _one_f_one_b(mbs, warm) + [Op("W", mbs[p]) for p in perm]
    elif kind == "1f1b_deferred_w":
        ops = _one_f_one_b(mbs, warm) + [Op("W", m) for m in mbs]
    elif kind == "coupled":
        ops = []
        for m in mbs:
            ops += [Op("F", m), Op("B", m), Op("W", m)]
    else:
        raise ValueError(f"unknown schedule {kind!r}")
    if with_step:
        ops.append(Op("STEP"))
    return ops
