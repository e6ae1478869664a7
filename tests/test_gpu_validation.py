"""Post-step validation on the GPU (section 5): gradient check, optimizer skip
and AdamW rollback; and selective decoupling under a stash limit (section
3.2), through the C ABI, against the fp64 oracle."""
import numpy as np
import pytest

import oracle
from synth import MB, gen_dy, gen_params, gen_x, get_config, op_list
from tests.conftest import compare_grads, rel_l2
from tests.gpu_harness import log, run_gpu, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    import paper_2405_14009_amd  # noqa: F401
    yield


def _iteration(cfg):
    return op_list(cfg, with_step=False)


def _state(stage):
    from paper_2405_14009_amd import RC_READ_ADAM_M, RC_READ_ADAM_V, RC_READ_PARAM
    return (stage.read_all(RC_READ_PARAM), stage.read_all(RC_READ_ADAM_M),
            stage.read_all(RC_READ_ADAM_V))


def _close(a, b, tol):
    for la, lb in zip(a, b):
        for x, y in zip(la, lb):
            if np.linalg.norm(y) == 0:
                assert np.abs(x).max() <= tol * 1e-3, np.abs(x).max()
            else:
                assert rel_l2(x, y) <= tol, rel_l2(x, y)


@pytest.mark.parametrize("name", ["small_f32", "small_bf16"])
def test_rollback_restores_the_state_before_the_step(name):
    cfg = get_config(name)
    log(f"[rollback] {name}")
    from paper_2405_14009_amd import Stage
    st = Stage.from_config(cfg)
    st.load_params(gen_params(cfg))
    run_gpu(cfg, _iteration(cfg), stage=st, read_state=False, keep_outputs=False)
    st.optimizer_step()                      # t = 1
    ops2 = _iteration(cfg)
    run_gpu(cfg, ops2, stage=st, read_state=False, keep_outputs=False)
    before = _state(st)
    x0 = to_device(gen_x(cfg, 0), cfg.dtype)
    st.optimizer_step(grad_scale=0.5)        # t = 2
    stepped = _state(st)
    st.optimizer_rollback()
    after = _state(st)
    _close(after[0], before[0], 1e-6)        # parameters: fp32 rounding of the inverse
    _close(after[1], before[1], 1e-5)
    _close(after[2], before[2], 1e-5)
    st.forward(MB(0), x0)                    # next iteration runs on the restored weights
    with pytest.raises(Exception):
        st.optimizer_rollback()              # nothing to undo any more
    log(f"[rollback] {name}: restored within tolerance; step moved params by "
        f"{max(rel_l2(s, b) for ls, lb in zip(stepped[0], before[0]) for s, b in zip(ls, lb)):.2e}")
    st.close()


def test_step_after_rollback_starts_a_new_iteration():
    """Rolling back the first step restores the zero moments exactly; the next
    step belongs to a new iteration (no weight pass yet: zero gradient, pure
    decay), as in the oracle."""
    cfg = get_config("small_bf16")
    from paper_2405_14009_amd import RC_OP_ROLLBACK, RC_OP_STEP, Stage
    st = Stage.from_config(cfg)
    st.load_params(gen_params(cfg))
    run_gpu(cfg, _iteration(cfg), stage=st, read_state=False, keep_outputs=False)
    st.optimizer_step()
    st.optimizer_rollback()
    _, m, v = _state(st)
    assert all(not np.any(t) for layer in m + v for t in layer)
    st.optimizer_step()
    again = _state(st)
    o = oracle.OracleStage(cfg, gen_params(cfg))
    o.optimizer_step()  # from the initial state with zero gradient
    for l in range(cfg.layers):
        for p in range(12):
            assert rel_l2(again[0][l][p], o.params[l][p]) < 1e-6
            assert not np.any(again[1][l][p]) and not np.any(again[2][l][p])
    assert [r[1] for r in st.op_log()[-3:]] == [RC_OP_STEP, RC_OP_ROLLBACK, RC_OP_STEP]
    st.close()


def test_skip_leaves_parameters_and_step_count():
    cfg = get_config("small_f32")
    from paper_2405_14009_amd import Stage
    st = Stage.from_config(cfg)
    st.load_params(gen_params(cfg))
    before = _state(st)
    run_gpu(cfg, _iteration(cfg), stage=st, read_state=False, keep_outputs=False)
    st.optimizer_skip()
    after = _state(st)
    for la, lb in zip(after, before):
        for x, y in zip(la, lb):
            for u, v in zip(x, y):
                assert np.array_equal(u, v)
    # the next step is still step 1: same result as the oracle's first step
    g = run_gpu(cfg, _iteration(cfg) + [op_list(cfg)[-1]], stage=st, read_state=True, keep_outputs=False)
    o = oracle.run_oplist(cfg)
    h = cfg.hidden
    keep = np.r_[0:h, 2 * h:3 * h]   # the K block of b_qkv has an exactly zero gradient: its
    for l in range(cfg.layers):      # first update is the sign of rounding noise on both sides
        for p in range(12):
            a, b = g.params[l][p], o.stage.params[l][p]
            if p == 3:
                a, b = a[keep], b[keep]
            assert rel_l2(a, b) < 1e-5
    st.close()


@pytest.mark.parametrize("name", ["small_f32", "small_bf16"])
def test_grad_check_against_oracle(name):
    cfg = get_config(name)
    from paper_2405_14009_amd import Stage
    st = Stage.from_config(cfg)
    st.load_params(gen_params(cfg))
    assert st.grad_check() == (0.0, 0)
    run_gpu(cfg, _iteration(cfg), stage=st, read_state=False, keep_outputs=False)
    o = oracle.OracleStage(cfg, gen_params(cfg))
    for op in _iteration(cfg):
        if op.kind == "F":
            o.forward(op.mb, gen_x(cfg, op.mb.j, op.mb.k))
        elif op.kind == "B":
            o.backward_input(op.mb, gen_dy(cfg, op.mb.j, op.mb.k))
        else:
            o.backward_weight(op.mb)
    ss, bad = st.grad_check(0.5)
    ss_o, bad_o = o.grad_check(0.5)
    tol = 2e-5 if cfg.dtype == "f32" else 4e-2
    log(f"[grad_check] {name}: gpu {ss:.6e} oracle {ss_o:.6e}")
    assert bad == 0 and bad_o == 0 and abs(ss - ss_o) <= tol * ss_o
    assert st.grad_check(0.5) == (ss, bad)   # bitwise reproducible
    st.optimizer_step()
    assert st.grad_check(0.5) == (ss, bad)   # right after the step: the gradient it used
    st.close()


def test_grad_check_counts_nonfinite_and_skip_keeps_weights():
    cfg = get_config("small_f32").with_(n_mb=1, schedule="coupled")
    from paper_2405_14009_amd import Stage
    st = Stage.from_config(cfg)
    st.load_params(gen_params(cfg))
    before = _state(st)
    dy = gen_dy(cfg, 0).copy()
    dy[0, 3, 5] = np.nan
    x = to_device(gen_x(cfg, 0), cfg.dtype)
    st.forward(MB(0), x)
    st.backward_input(MB(0), to_device(dy, cfg.dtype))
    st.backward_weight(MB(0))
    ss, bad = st.grad_check()
    o = oracle.OracleStage(cfg, gen_params(cfg))
    o.forward(MB(0), gen_x(cfg, 0))
    o.backward_input(MB(0), dy)
    o.backward_weight(MB(0))
    ss_o, bad_o = o.grad_check()
    log(f"[grad_check] planted NaN: gpu {bad} non-finite, oracle {bad_o}")
    assert bad > 0 and bad_o > 0
    st.optimizer_skip()
    after = _state(st)
    for x1, y1 in zip(after[0], before[0]):
        for u, v in zip(x1, y1):
            assert np.array_equal(u, v)
    st.close()


@pytest.mark.parametrize("slots", [1, 0])
def test_executor_under_a_stash_limit_matches_the_deferred_run(slots):
    """Coupled backward passes and early weight passes only reorder the
    gradient sum: same gradients (fp32 sums in another order: <= 1e-6) and the
    same outputs as the fully deferred run, with the stash kept under the
    limit; and the limited run's outputs and gradients match the oracle's run
    of the same op list."""
    from paper_2405_14009_amd import RC_READ_GRAD, Stage
    from paper_2405_14009_amd.executor import execute
    cfg = get_config("small_bf16").with_(n_mb=6)
    ops = op_list(cfg, with_step=False)
    xs = {(mb.j, mb.k): to_device(gen_x(cfg, mb.j, mb.k), cfg.dtype) for mb in
          [o.mb for o in ops if o.kind == "F"]}
    dys = {k: to_device(gen_dy(cfg, *k), cfg.dtype) for k in xs}

    def run(limit):
        st = Stage.from_config(cfg)
        st.load_params(gen_params(cfg))
        outs = {}
        rep = execute(st, ops, x_fn=lambda mb: xs[mb], dy_fn=lambda mb: dys[mb], stash_limit=limit,
                      on_output=lambda kind, mb, t: outs.__setitem__((kind,) + mb, t.float().cpu().numpy()))
        g = st.read_all(RC_READ_GRAD)
        st.close()
        return rep, g, outs

    ref_rep, ref_g, ref_out = run(0)
    a = Stage.from_config(cfg, dry_run=True).stash_account()
    limit = (cfg.warmup + 1) * a["a_f"] + slots * a["s_w"]
    rep, g, out = run(limit)
    log(f"[stash limit] slots={slots}: peak {rep.peak} <= {limit}; coupled {len(rep.coupled)}, "
        f"early {len(rep.flushed)}; unlimited peak {ref_rep.peak}")
    assert rep.peak <= limit < ref_rep.peak
    assert rep.coupled or rep.flushed
    for k in ref_out:
        assert np.array_equal(out[k], ref_out[k]), k
    for l in range(cfg.layers):
        for p in range(12):
            assert rel_l2(g[l][p], ref_g[l][p]) < 1e-6, (l, p)
    o = oracle.run_oplist(cfg, ops)
    for mb in o.y:
        assert rel_l2(out[("F",) + mb], o.y[mb]) < 2e-2, ("y", mb)
        assert rel_l2(out[("B",) + mb], o.dx[mb]) < 2e-2, ("dx", mb)
    worst = compare_grads(cfg, g, o.grads, 2e-2)
    log(f"[stash limit] slots={slots}: worst gradient rel-L2 against the oracle {worst:.2e}")


def test_simulated_peer_op_list_drives_the_stage():
    """The schedule simulator's op list of a peer that absorbs a failed
    worker's micro-batches (3 pipelines x 4 stages, W_1_2 failed, Decoupled
    BackProp) runs through the executor on the GPU: op log and gradients
    match the oracle executing the same list."""
    from paper_2405_14009_amd import Stage
    from paper_2405_14009_amd.executor import execute
    from paper_2405_14009_amd.planner import simulate
    from synth.schedules import Op
    sim = simulate(3, 4, 6, failed=[(1, 2)], decoupled=True)
    mine = sim.worker_ops(0, 2)
    ops = [Op(o.kind, MB(o.j, o.k)) for o in mine] + [Op("STEP")]
    n = sum(1 for o in mine if o.kind == "F")
    assert n == 9 and any(o.k == 1 for o in mine)
    cfg = get_config("small_f32").with_(n_mb=n, max_stashed_mb=n, max_inflight_mb=n)
    st = Stage.from_config(cfg, pipeline_id=0)
    st.load_params(gen_params(cfg))
    g = run_gpu(cfg, [o for o in ops if o.kind != "STEP"], stage=st, read_state=True, keep_outputs=False)
    o = oracle.run_oplist(cfg, ops=ops)
    assert g.log == [tuple(r) for r in o.stage.log][:-1]
    for l in range(cfg.layers):
        for p in range(12):
            assert rel_l2(g.grads[l][p], o.grads[l][p]) < 1e-5
    st.close()
    # the same list through the executor (batched deferred weight passes)
    st = Stage.from_config(cfg, pipeline_id=0)
    st.load_params(gen_params(cfg))
    rep = execute(st, ops, x_fn=lambda mb: to_device(gen_x(cfg, *mb), cfg.dtype),
                  dy_fn=lambda mb: to_device(gen_dy(cfg, *mb), cfg.dtype))
    assert st.op_log() == [tuple(r) for r in o.stage.log]
    log(f"[simulated peer] {len(mine)} ops, {rep.weight_calls} weight-pass calls")
    st.close()
