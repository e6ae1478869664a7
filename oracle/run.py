"""Drive an OracleStage through an op list on seeded inputs (test infrastructure)."""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

from synth import gen_dy, gen_params, gen_x, op_list
from .stage import AdamHP, OracleStage


@dataclass
class OracleRun:
    y: Dict[Tuple[int, int], np.ndarray] = field(default_factory=dict)
    dx: Dict[Tuple[int, int], np.ndarray] = field(default_factory=dict)
    grads: Optional[list] = None           # gradients after the last W (before the step)
    stage: Optional[OracleStage] = None    # params/m/v after the step, op log


def run_oplist(cfg, ops=None, params=None, hp: Optional[AdamHP] = None, x_fn=None, dy_fn=None,
               stage_index: int = 0, pipeline_id: int = 0) -> OracleRun:
    """Execute ``ops`` (default: the config's op list) on the oracle.

    ``x_fn(j, k)`` / ``dy_fn(j, k)`` override the seeded inputs."""
    ops = op_list(cfg) if ops is None else ops
    params = gen_params(cfg) if params is None else params
    x_fn = x_fn or (lambda j, k: gen_x(cfg, j, k))
    dy_fn = dy_fn or (lambda j, k: gen_dy(cfg, j, k))
    st = OracleStage(cfg, params, hp=hp, stage_index=stage_index, pipeline_id=pipeline_id)
    out = OracleRun(stage=st)
    for op in ops:
        if op.kind == "F":
            out.y[tuple(op.mb)] = st.forward(op.mb, x_fn(op.mb.j, op.mb.k))
        elif op.kind == "B":
            out.dx[tuple(op.mb)] = st.backward_input(op.mb, dy_fn(op.mb.j, op.mb.k))
        elif op.kind == "W":
            st.backward_weight(op.mb)
        elif op.kind == "STEP":
            out.grads = [[g.copy() for g in layer] for layer in st.grads]
            st.optimizer_step()
    if out.grads is None:
        out.grads = [[g.copy() for g in layer] for layer in st.grads]
    return out
