import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (HIP device) and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def rel_l2(a, b) -> float:
    """||a - b|| / ||b|| in fp64 (absolute norm when ||b|| == 0)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    d = np.linalg.norm(a - b)
    return float(d / nb) if nb > 0 else float(d)


def compare_grads(cfg, got, ref, t):
    """Every gradient of every layer (the K block of the QKV bias, whose exact
    value is zero, by its norm against the V block's); returns the worst."""
    h, worst = cfg.hidden, {}
    for l in range(cfg.layers):
        for p in range(12):
            if p == 3:
                keep = np.r_[0:h, 2 * h:3 * h]
                worst[(l, p)] = rel_l2(got[l][p][keep], ref[l][p][keep])
                ratio = np.linalg.norm(got[l][p][h:2 * h]) / np.linalg.norm(got[l][p][2 * h:])
                assert ratio < t, ("|grad b_k| / |grad b_v|", l, ratio)
            else:
                worst[(l, p)] = rel_l2(got[l][p], ref[l][p])
    bad = {k: v for k, v in worst.items() if v > t}
    assert not bad, bad
    return max(worst.values())
