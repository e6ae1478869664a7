"""The no-allocation entry point rc_stage_create_static (work memory in the
library's own per-device array instead of a caller arena) gives exactly the
results of rc_stage_create on the same op list, on two handles in a row, the
second with a smaller workload (its work memory then starts with what the
first left there)."""
import numpy as np
import pytest

from synth import get_config
from tests.gpu_harness import log, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    import paper_2405_14009_amd  # noqa: F401  (fails loudly if the library is missing)
    yield


def _same(a, b, what):
    assert a.log == b.log, what
    for mb in b.y:
        assert np.array_equal(a.y[mb], b.y[mb]), (what, "y", mb)
        assert np.array_equal(a.dx[mb], b.dx[mb]), (what, "dx", mb)
    for name in ("grads", "params", "m", "v"):
        for l, (la, lb) in enumerate(zip(getattr(a, name), getattr(b, name))):
            for p, (x, y) in enumerate(zip(la, lb)):
                assert np.array_equal(x, y), (what, name, l, p)


def test_static_work_matches_caller_work():
    from paper_2405_14009_amd import Stage
    big = get_config("small_bf16")
    small = big.with_(seq=136, micro_batch=1, n_mb=2, rerouted=(1,), layers=1)
    assert Stage.from_config(small, dry_run=True).work_bytes < Stage.from_config(big, dry_run=True).work_bytes
    for cfg in (big, small):
        log(f"[no-alloc] {cfg.name} s={cfg.seq} b={cfg.micro_batch} L={cfg.layers} n_mb={cfg.n_mb}")
        got = run_gpu(cfg, static_work=True)
        ref = run_gpu(cfg)
        _same(got, ref, (cfg.seq, cfg.micro_batch))
