"""Drive the HIP stage through the C ABI on seeded inputs and collect what
the parity tests compare (test infrastructure)."""
from __future__ import annotations

import sys
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

from synth import bf16_bits, bf16_bits_to_f32, gen_dy, gen_params, gen_x, op_list


def to_device(a: np.ndarray, dtype: str):
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(bf16_bits(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to("cuda")


def to_host(t) -> np.ndarray:
    import torch
    if t.dtype == torch.bfloat16:
        return bf16_bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    return t.float().cpu().numpy().astype(np.float64)


@dataclass
class GpuRun:
    y: Dict[Tuple[int, int], np.ndarray] = field(default_factory=dict)
    dx: Dict[Tuple[int, int], np.ndarray] = field(default_factory=dict)
    grads: Optional[list] = None
    params: Optional[list] = None
    m: Optional[list] = None
    v: Optional[list] = None
    log: Optional[list] = None


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def run_gpu(cfg, ops=None, params=None, x_fn=None, dy_fn=None, stage=None, read_state=True,
            keep_outputs=True, **stage_kw) -> GpuRun:
    """Execute ``ops`` on a fresh HIP stage (or ``stage``) and collect outputs."""
    from paper_2405_14009_amd import (RC_READ_ADAM_M, RC_READ_ADAM_V, RC_READ_GRAD, RC_READ_PARAM,
                                      Stage)
    ops = op_list(cfg) if ops is None else ops
    x_fn = x_fn or (lambda j, k: gen_x(cfg, j, k))
    dy_fn = dy_fn or (lambda j, k: gen_dy(cfg, j, k))
    own = stage is None
    if own:
        stage = Stage.from_config(cfg, **stage_kw)
        stage.load_params(gen_params(cfg) if params is None else params)
    out = GpuRun()
    for op in ops:
        if op.kind == "F":
            y = stage.forward(op.mb, to_device(x_fn(op.mb.j, op.mb.k), cfg.dtype))
            if keep_outputs:
                out.y[tuple(op.mb)] = to_host(y)
        elif op.kind == "B":
            dx = stage.backward_input(op.mb, to_device(dy_fn(op.mb.j, op.mb.k), cfg.dtype))
            if keep_outputs:
                out.dx[tuple(op.mb)] = to_host(dx)
        elif op.kind == "W":
            stage.backward_weight(op.mb)
        elif op.kind == "W*":          # batched weight pass over a list of micro-batches
            stage.backward_weight_many(op.mb)
        else:
            if read_state:
                out.grads = stage.read_all(RC_READ_GRAD)
            stage.optimizer_step()
    stage.synchronize()
    if read_state:
        if out.grads is None:
            out.grads = stage.read_all(RC_READ_GRAD)
        out.params = stage.read_all(RC_READ_PARAM)
        out.m = stage.read_all(RC_READ_ADAM_M)
        out.v = stage.read_all(RC_READ_ADAM_V)
    out.log = stage.op_log()
    if own:
        stage.close()
    return out
