"""Plain CPU reference of the schedule-side pieces of ReCycle (test
infrastructure, like the rest of this package).

* ``cost`` / ``failure_normalization``: Failure Normalization (section 4.2.1,
  Algorithm 1), a dynamic programme over stages that assigns F failures to
  pipeline stages.
* ``bubble_capacity``: the idle-slot count of the 1F1B schedule that Adaptive
  Pipelining uses for re-routed work (section 3.1).
* ``simulate``: a unit-slot simulator of DP data-parallel pipelines of PP
  stages running 1F1B over MB micro-batches each, with failed workers'
  micro-batches re-routed round-robin to their peers (section 3.1), the
  backward pass optionally split into B_input and a deferred B_weight
  (section 3.2), and optionally a staggered optimizer (section 3.3).

Readings (where the paper is silent or garbled):
* COST: the printed ``min(0, MB f 3 - (DP - f)(PP - 1) 3)`` is never
  positive; read as ``max(0, ...)``: extra slots = re-routed work (3 slots
  per micro-batch) minus the peers' bubbles (3 (PP-1) per worker).
* argmin ties in Algorithm 1 go to the larger x, i.e. failures move to later
  stages (the paper's single-failure example lands on the last stage).
* A stage can lose at most DP - 1 of its DP workers.
* Slots: F = 1, B_input = 1, B_weight = 1; a coupled backward = 2.
* Worker policy: a ready backward first, then a ready forward, then
  (decoupled) a deferred weight pass, oldest first; ties in micro-batch order
  (origin pipeline, then index).  No cap on micro-batches between F and B
  unless ``inflight_cap`` is given (1F1B's textbook depth is PP - i).  This
  plain rule reproduces the paper's running example (DP 3, PP 4, 6
  micro-batches): 27 slots and 9 bubbles per worker fault-free, 36 slots with
  one failed worker and a coupled backward, 29 with Decoupled BackProp.
* Synchronous optimizer: iteration n+1 starts when every worker has finished
  iteration n.  Staggered: stage i starts iteration n+1 once every worker of
  stage i has finished iteration n (the per-stage all-reduce and step take
  no slot).
"""
from __future__ import annotations

import itertools
from typing import Dict, List, Sequence, Tuple


def cost(dp: int, pp: int, mb: int, f: int) -> int:
    """Extra slots for f failures on one stage (Algorithm 1's COST)."""
    if f <= 0:
        return 0
    return max(0, mb * f * 3 - (dp - f) * (pp - 1) * 3)


def failure_normalization(dp: int, pp: int, mb: int, failures: int) -> Tuple[List[int], int]:
    """Algorithm 1: (failures per stage, total overhead).  O[i][f] is the least
    overhead of f failures on stages 0..i and A[i][f] its assignment."""
    if failures < 0 or failures > pp * (dp - 1):
        raise ValueError("more failures than the pipeline can survive")
    INF = float("inf")
    O = [[INF] * (failures + 1) for _ in range(pp)]
    A: List[List[List[int]]] = [[[] for _ in range(failures + 1)] for _ in range(pp)]
    for i in range(pp):
        for f in range(failures + 1):
            if i == 0:
                if f <= dp - 1:
                    O[0][f] = cost(dp, pp, mb, f)
                    A[0][f] = [f]
                continue
            best, bx = INF, None
            for x in range(min(f, dp - 1) + 1):
                c = O[i - 1][f - x] + cost(dp, pp, mb, x)
                if c <= best:          # ties: the larger x (later stage)
                    best, bx = c, x
            O[i][f] = best
            if bx is not None and best < INF:
                A[i][f] = A[i - 1][f - bx] + [bx]
    return A[pp - 1][failures], int(O[pp - 1][failures])


def failure_normalization_brute_force(dp: int, pp: int, mb: int, failures: int) -> int:
    """Least total overhead over every assignment of failures to stages."""
    best = None
    for a in itertools.product(range(dp), repeat=pp):
        if sum(a) == failures:
            c = sum(cost(dp, pp, mb, x) for x in a)
            best = c if best is None else min(best, c)
    return best


def bubble_capacity(pp: int, dp: int) -> int:
    """Idle slots per iteration that the peers of a pipeline offer: each of
    the DP workers of a stage has 3 (PP - 1) bubbles in 1F1B (F = 1 slot,
    B = 2 slots)."""
    return 3 * (pp - 1) * dp


def round_robin_reroute(dp: int, failed: Sequence[Tuple[int, int]], mb: int) -> Dict[Tuple[int, int, int], int]:
    """Executing pipeline k_s of micro-batch (stage i, index j, origin k):
    the failed worker's micro-batches go round-robin to the alive peers of its
    stage in increasing pipeline order."""
    dead = set(failed)
    out = {}
    for (k, i) in failed:
        alive = [p for p in range(dp) if (p, i) not in dead]
        for n, j in enumerate(range(mb)):
            out[(i, j, k)] = alive[n % len(alive)]
    return out


def simulate(dp: int, pp: int, mb: int, failed: Sequence[Tuple[int, int]] = (),
             decoupled: bool = False, staggered: bool = False, iterations: int = 1,
             inflight_cap=None):
    """Unit-slot simulation.  Returns (makespan, per-worker busy slots, per-worker
    op list [(slot, kind, iteration, i, j, k)], per-iteration end slot)."""
    dead = set(failed)
    route = round_robin_reroute(dp, failed, mb)

    def runner(i, j, k):
        return route.get((i, j, k), k)

    # per micro-batch per stage: completion slot of F, B (B_input), W
    done_f: Dict[tuple, int] = {}
    done_b: Dict[tuple, int] = {}
    done_w: Dict[tuple, int] = {}
    workers = [(k, i) for k in range(dp) for i in range(pp) if (k, i) not in dead]
    busy = {w: 0 for w in workers}
    log = {w: [] for w in workers}
    bdur = 1 if decoupled else 2
    iter_end = []
    t = 0
    start_of = {w: 0 for w in workers}
    for it in range(iterations):
        mine = {w: [(it, i, j, k) for k in range(dp) for j in range(mb) for i in [w[1]]
                    if runner(w[1], j, k) == w[0]] for w in workers}
        free_at = {w: max(t, start_of[w]) for w in workers}
        pending = {w: list(mine[w]) for w in workers}
        inflight = {w: set() for w in workers}
        deferred = {w: [] for w in workers}
        remaining = sum(len(v) for v in pending.values()) * (3 if decoupled else 2)
        now = min(free_at.values())
        while remaining:
            started = False
            for w in sorted(workers):
                if free_at[w] > now:
                    continue
                i = w[1]
                op = None
                # backward first
                for key in sorted(inflight[w], key=lambda q: (q[3], q[2])):
                    _, _, j, k = key
                    ready = key in done_f and done_f[key] <= now
                    if i < pp - 1:
                        nxt = (it, i + 1, j, k)
                        ready = ready and nxt in done_b and done_b[nxt] <= now
                    if ready:
                        op = ("B", key)
                        break
                if op is None and (inflight_cap is None or len(inflight[w]) < inflight_cap(i)):
                    for key in sorted(pending[w], key=lambda q: (q[3], q[2])):
                        _, _, j, k = key
                        prev = (it, i - 1, j, k)
                        if i == 0 or (prev in done_f and done_f[prev] <= now):
                            op = ("F", key)
                            break
                if op is None and deferred[w]:
                    op = ("W", deferred[w][0])
                if op is None:
                    continue
                kind, key = op
                if kind == "F":
                    pending[w].remove(key)
                    inflight[w].add(key)
                    done_f[key] = now + 1
                    free_at[w] = now + 1
                elif kind == "B":
                    inflight[w].remove(key)
                    done_b[key] = now + bdur
                    free_at[w] = now + bdur
                    if decoupled:
                        deferred[w].append(key)
                    else:
                        done_w[key] = now + bdur
                else:
                    deferred[w].remove(key)
                    done_w[key] = now + 1
                    free_at[w] = now + 1
                remaining -= 1
                started = True
                busy[w] += 1 if kind != "B" else bdur
                log[w].append((now, kind, it, key[1], key[2], key[3]))
            if not started and all(free_at[w] <= now for w in workers):
                raise ValueError("schedule cannot make progress")
            now += 1
        end = max(free_at.values())
        iter_end.append(end)
        if staggered:
            for i in range(pp):
                stage_end = max(free_at[w] for w in workers if w[1] == i)
                for w in workers:
                    if w[1] == i:
                        start_of[w] = stage_end
            t = min(start_of.values())
        else:
            t = end
            for w in workers:
                start_of[w] = end
    return max(iter_end), busy, log, iter_end
