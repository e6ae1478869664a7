"""Seeded per-tensor random streams and bf16 round-to-nearest-even.

Every tensor has its own stream, ``numpy.random.default_rng([seed, stream,
index])``, so tensors can be generated lazily, in any order, and identically
by the oracle and by the GPU harness:

* stream 1: parameters, index = layer * 16 + param_id
* stream 2: stage input x of micro-batch (j, k), index = k * 65536 + j
* stream 3: upstream gradient dy of micro-batch (j, k), same index
* stream 4: the order in which deferred weight passes are issued

Values are ``standard_normal(float32) * std``; for bf16 workloads they are
rounded to bf16 (round to nearest, ties to even) so that both sides consume
exactly the same numbers.
"""
from __future__ import annotations

import numpy as np

# Parameter order inside one pre-LN transformer layer; the id is the index.
PARAM_NAMES = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
               "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2")


def PARAM_SHAPES(h: int, f: int):
    """Shapes of the 12 parameters of a layer, in PARAM_NAMES order.

    Linear weights are stored [in, out] (y = x @ W); the fused QKV weight is
    [h, 3h] with column blocks Q | K | V.
    """
    return ((h,), (h,), (h, 3 * h), (3 * h,), (h, h), (h,),
            (h,), (h,), (h, f), (f,), (f, h), (h,))


def is_matrix_param(pid: int) -> bool:
    return pid in (2, 4, 8, 10)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) of float32 values that are bf16-representable."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal(seed: int, stream: int, index: int, shape, std: float) -> np.ndarray:
    g = np.random.default_rng([seed, stream, index])
    out = g.standard_normal(size=shape, dtype=np.float32)
    out *= np.float32(std)
    return out


def _finish(a: np.ndarray, dtype: str) -> np.ndarray:
    return round_bf16(a) if dtype == "bf16" else a


def gen_param(cfg, layer: int, pid: int) -> np.ndarray:
    """Initial value of parameter ``pid`` of ``layer`` as float32.

    Linear weights ~ N(0, w_std) (second argument = standard deviation); biases
    0, LN gamma 1, beta 0.  With ``cfg.perturbed`` the vectors get N(0, 0.02)
    offsets so that the bias/affine paths are exercised by tests.
    """
    shape = PARAM_SHAPES(cfg.hidden, cfg.ffn)[pid]
    if is_matrix_param(pid):
        a = _normal(cfg.seed, 1, layer * 16 + pid, shape, cfg.w_std)
    else:
        base = 1.0 if pid in (0, 6) else 0.0
        if cfg.perturbed:
            a = _normal(cfg.seed, 1, layer * 16 + pid, shape, 0.02) + np.float32(base)
        else:
            a = np.full(shape, base, dtype=np.float32)
    return _finish(a, cfg.dtype)


def gen_params(cfg):
    """All parameters: list over layers of lists over PARAM_NAMES (float32)."""
    return [[gen_param(cfg, l, p) for p in range(len(PARAM_NAMES))] for l in range(cfg.layers)]


def gen_x(cfg, j: int, k: int = 0, seq: int | None = None) -> np.ndarray:
    """Stage input activations of micro-batch (j, k): [b, s, h] ~ N(0, x_std)."""
    a = _normal(cfg.seed, 2, k * 65536 + j, (cfg.micro_batch, cfg.seq, cfg.hidden), cfg.x_std)
    if seq is not None:
        a = np.ascontiguousarray(a[:, :seq])
    return _finish(a, cfg.dtype)


def gen_dy(cfg, j: int, k: int = 0, keep_prefix: int | None = None) -> np.ndarray:
    """Upstream gradient of micro-batch (j, k): [b, s, h] ~ N(0, dy_std).

    ``keep_prefix=t0`` zeroes every position >= t0 (a valid input of the same
    shape; with causal attention the resulting dx and weight gradients depend
    only on the first t0 positions).
    """
    a = _normal(cfg.seed, 3, k * 65536 + j, (cfg.micro_batch, cfg.seq, cfg.hidden), cfg.dy_std)
    if keep_prefix is not None:
        a[:, keep_prefix:] = 0.0
    return _finish(a, cfg.dtype)


def wshuffle_perm(cfg, n: int) -> np.ndarray:
    return np.random.default_rng([cfg.seed, 4, 0]).permutation(n)
