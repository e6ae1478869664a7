"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test ties the oracle to something other than itself:

* central finite differences of  J = sum(y * dy)  (pins the whole backward,
  both the input-gradient pass and the weight-gradient pass, to the forward);
* an independent torch fp64 build of the same block from library routines
  (layer_norm, scaled_dot_product_attention, tanh GeLU, linear) and torch
  autograd (pins the forward and the backward);
* torch.optim.AdamW in fp64 and the t = 1 closed form (pins the optimizer);
* invariants the paper states: decoupled B_input + B_weight equals the coupled
  backward (Decoupled BackProp, section 3.2); gradients do not depend on the
  order of deferred weight passes nor on which peer runs a re-routed
  micro-batch (Adaptive Pipelining, section 3.1: the computation of the
  iteration is unchanged); B_input precedes B_weight (same-stage constraint
  of the schedule MILP);
* mathematical invariants: causality, micro-batch split, linearity in dy,
  LayerNorm and softmax backward orthogonality, s = 1 special case.

The mutation tests at the end plant a mistake in the oracle (on the CPU) and
check that a pin catches it.
"""
import copy
import itertools

import numpy as np
import pytest

import oracle
from oracle import stage as ost
from synth import MB, StageConfig, gen_dy, gen_params, gen_x, get_config, op_list
from tests.conftest import rel_l2

F64 = np.float64


def small_cfg(**kw):
    base = dict(name="pin", layers=2, hidden=8, heads=2, ffn=32, seq=5, micro_batch=2,
                causal=True, dtype="f32", n_mb=2, perturbed=True, schedule="coupled")
    base.update(kw)
    return StageConfig(**base)


def params64(cfg):
    return [[p.astype(F64) for p in layer] for layer in gen_params(cfg)]


def shape_of(cfg):
    return ost.LayerShape(cfg.heads, cfg.causal, cfg.ln_eps)


def decoupled(cfg, params, x, dy):
    shp = shape_of(cfg)
    y, caches = ost.stage_forward(x, params, shp)
    dx, stashes = ost.stage_backward_input(dy, caches, params)
    grads = ost.stage_backward_weight(stashes)
    return y, dx, grads


# ---------------------------------------------------------------------------
# Finite differences
# ---------------------------------------------------------------------------

def fd_check(cfg, step=1e-6):
    params = params64(cfg)
    x = gen_x(cfg, 0).astype(F64)
    dy = gen_dy(cfg, 0).astype(F64) * 100.0
    shp = shape_of(cfg)

    def J(xx, pp):
        return float((ost.stage_forward(xx, pp, shp)[0] * dy).sum())

    _, dx, grads = decoupled(cfg, params, x, dy)
    num_dx = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        xp = x.copy(); xp[i] += step
        xm = x.copy(); xm[i] -= step
        num_dx[i] = (J(xp, params) - J(xm, params)) / (2 * step)
    errs = {"dx": rel_l2(dx, num_dx)}
    for l in range(cfg.layers):
        for p in range(12):
            t = params[l][p]
            num = np.zeros_like(t)
            flat = t.reshape(-1)
            nflat = num.reshape(-1)
            for e in range(flat.size):
                old = flat[e]
                flat[e] = old + step
                jp = J(x, params)
                flat[e] = old - step
                jm = J(x, params)
                flat[e] = old
                nflat[e] = (jp - jm) / (2 * step)
            errs[(l, p)] = rel_l2(grads[l][p], num)
    return errs


@pytest.mark.parametrize("causal", [True, False])
def test_finite_differences(causal):
    errs = fd_check(small_cfg(causal=causal))
    worst = max(errs.values())
    assert worst < 1e-6, {k: v for k, v in errs.items() if v >= 1e-6}


# ---------------------------------------------------------------------------
# Independent torch fp64 build of the same layer (library routines + autograd)
# ---------------------------------------------------------------------------

def torch_stage(cfg, params, x, dy):
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    h, a = cfg.hidden, cfg.heads
    d = h // a
    tp = [[torch.tensor(p, dtype=torch.float64, requires_grad=True) for p in layer] for layer in params]
    tx = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    z = tx
    for layer in tp:
        g1, be1, wqkv, bqkv, wo, bo, g2, be2, w1, b1, w2, b2 = layer
        A = F.layer_norm(z, (h,), g1, be1, eps=cfg.ln_eps)
        # torch.nn.functional.linear takes weight as [out, in]
        q = F.linear(A, wqkv[:, 0:h].t(), bqkv[0:h])
        k = F.linear(A, wqkv[:, h:2 * h].t(), bqkv[h:2 * h])
        v = F.linear(A, wqkv[:, 2 * h:].t(), bqkv[2 * h:])
        b_, s_ = q.shape[0], q.shape[1]
        heads = lambda t: t.reshape(b_, s_, a, d).transpose(1, 2)
        o = F.scaled_dot_product_attention(heads(q), heads(k), heads(v), is_causal=cfg.causal)
        o = o.transpose(1, 2).reshape(b_, s_, h)
        H = z + F.linear(o, wo.t(), bo)
        C = F.layer_norm(H, (h,), g2, be2, eps=cfg.ln_eps)
        G = F.gelu(F.linear(C, w1.t(), b1), approximate="tanh")
        z = H + F.linear(G, w2.t(), b2)
    (z * torch.tensor(dy, dtype=torch.float64)).sum().backward()
    return (z.detach().numpy(), tx.grad.numpy(),
            [[p.grad.numpy() for p in layer] for layer in tp])


@pytest.mark.parametrize("causal", [True, False])
def test_against_torch_autograd(causal):
    cfg = small_cfg(layers=2, hidden=64, heads=4, ffn=256, seq=33, causal=causal)
    params = params64(cfg)
    x = gen_x(cfg, 1).astype(F64)
    dy = gen_dy(cfg, 1).astype(F64)
    y, dx, grads = decoupled(cfg, params, x, dy)
    ty, tdx, tgrads = torch_stage(cfg, params, x, dy)
    assert rel_l2(y, ty) < 1e-12
    assert rel_l2(dx, tdx) < 1e-10
    for l in range(cfg.layers):
        for p in range(12):
            assert rel_l2(grads[l][p], tgrads[l][p]) < 1e-10, (l, p)


def test_tiny_config_against_torch():
    cfg = get_config("tiny_perturbed")
    params = params64(cfg)
    x = gen_x(cfg, 0).astype(F64)
    dy = gen_dy(cfg, 0).astype(F64)
    y, dx, grads = decoupled(cfg, params, x, dy)
    ty, tdx, tgrads = torch_stage(cfg, params, x, dy)
    assert rel_l2(y, ty) < 1e-12 and rel_l2(dx, tdx) < 1e-10
    assert max(rel_l2(grads[0][p], tgrads[0][p]) for p in range(12)) < 1e-10


# ---------------------------------------------------------------------------
# Invariants stated by the paper
# ---------------------------------------------------------------------------

def test_decoupled_equals_fused():
    for cfg in (small_cfg(), small_cfg(hidden=48, heads=3, ffn=96, seq=17, causal=False),
                get_config("tiny_perturbed")):
        params = params64(cfg)
        x = gen_x(cfg, 2).astype(F64)
        dy = gen_dy(cfg, 2).astype(F64)
        y, dx, grads = decoupled(cfg, params, x, dy)
        y2, caches = ost.stage_forward(x, params, shape_of(cfg))
        dx2, grads2 = ost.stage_backward_fused(dy, caches, params)
        assert np.array_equal(y, y2)
        assert rel_l2(dx, dx2) < 1e-12
        for l in range(cfg.layers):
            for p in range(12):
                assert rel_l2(grads[l][p], grads2[l][p]) < 1e-12


def _run_fb(cfg):
    st = oracle.OracleStage(cfg, gen_params(cfg))
    mbs = [MB(j, 1 if j in cfg.rerouted else 0) for j in range(cfg.n_mb)]
    for m in mbs:
        st.forward(m, gen_x(cfg, m.j, m.k))
    for m in mbs:
        st.backward_input(m, gen_dy(cfg, m.j, m.k))
    return st, mbs


def test_w_order_invariance_all_permutations_tiny():
    cfg = get_config("tiny_perturbed")
    st, mbs = _run_fb(cfg)
    ref = None
    for perm in itertools.permutations(range(len(mbs))):
        s2 = copy.deepcopy(st)
        for i in perm:
            s2.backward_weight(mbs[i])
        g = [np.concatenate([t.ravel() for t in layer]) for layer in s2.grads]
        if ref is None:
            ref = g
        for a, b in zip(g, ref):
            assert rel_l2(a, b) < 1e-12


def test_w_order_invariance_seeded_shuffle():
    cfg = small_cfg(n_mb=16, layers=1, hidden=32, heads=2, ffn=64, seq=9, micro_batch=1)
    st, mbs = _run_fb(cfg)
    a, b = copy.deepcopy(st), copy.deepcopy(st)
    for m in mbs:
        a.backward_weight(m)
    for i in np.random.default_rng([0, 4, 0]).permutation(16):
        b.backward_weight(mbs[i])
    for la, lb in zip(a.grads, b.grads):
        for ta, tb in zip(la, lb):
            assert rel_l2(ta, tb) < 1e-12


@pytest.mark.parametrize("policy", ["round_robin", "all_to_one", "random"])
def test_peer_reroute_invariance(policy):
    """DP = 3 replicas of a stage; pipeline 1 fails and its micro-batches are
    re-routed to the surviving peers (round-robin over alive peers is the
    paper's policy, ReRouteAct in section 5).  The sum of the peers' gradients
    equals the fault-free sum, and every micro-batch's y and dx are identical
    whichever peer executes it."""
    cfg = small_cfg(layers=1, hidden=16, heads=2, ffn=32, seq=6, micro_batch=1, n_mb=4)
    params = gen_params(cfg)
    dp = 3
    work = {k: [MB(j, k) for j in range(cfg.n_mb)] for k in range(dp)}

    def run(assign):
        outs, total = {}, None
        for ks, mbs in assign.items():
            st = oracle.OracleStage(cfg, params, pipeline_id=ks, max_stashed=99, max_inflight=99)
            for m in mbs:
                outs[("y", m)] = st.forward(m, gen_x(cfg, m.j, m.k))
            for m in mbs:
                outs[("dx", m)] = st.backward_input(m, gen_dy(cfg, m.j, m.k))
            for m in mbs:
                st.backward_weight(m)
            g = [np.concatenate([t.ravel() for t in layer]) for layer in st.grads]
            total = g if total is None else [a + b for a, b in zip(total, g)]
        return outs, total

    ff_out, ff_total = run(work)
    alive = [0, 2]
    failed = work[1]
    assign = {0: list(work[0]), 2: list(work[2])}
    rng = np.random.default_rng(7)
    for i, m in enumerate(failed):
        if policy == "round_robin":
            tgt = alive[i % len(alive)]
        elif policy == "all_to_one":
            tgt = alive[0]
        else:
            tgt = alive[int(rng.integers(len(alive)))]
        assign[tgt].append(m)
    rr_out, rr_total = run(assign)
    for key, val in ff_out.items():
        assert np.array_equal(val, rr_out[key]), key
    for a, b in zip(rr_total, ff_total):
        assert rel_l2(a, b) < 1e-12


def test_same_stage_dependency_and_error_table():
    cfg = small_cfg(n_mb=3, max_stashed_mb=2, max_inflight_mb=1)
    st = oracle.OracleStage(cfg, gen_params(cfg))
    x, dy = gen_x(cfg, 0), gen_dy(cfg, 0)
    m0, m1, m2 = MB(0), MB(1), MB(2)

    def code(fn, *a):
        with pytest.raises(oracle.StageError) as e:
            fn(*a)
        return e.value.code

    assert code(st.backward_input, m0, dy) == "BAD_STATE"      # B before F
    assert code(st.backward_weight, m0) == "BAD_STATE"         # W before B
    st.forward(m0, x)
    assert code(st.forward, m0, x) == "BAD_STATE"              # F twice
    assert code(st.backward_weight, m0) == "BAD_STATE"         # W before B
    assert code(st.forward, m1, x) == "OUT_OF_STASH"           # 1 in-flight slot
    st.backward_input(m0, dy)
    assert code(st.backward_input, m0, dy) == "BAD_STATE"      # B twice
    st.forward(m1, x)
    assert code(st.forward, m2, x) == "OUT_OF_STASH"           # 2 stash slots
    assert code(st.optimizer_step) == "BAD_STATE"              # pending W
    st.backward_weight(m0)
    assert code(st.backward_weight, m0) == "BAD_STATE"         # W twice
    assert code(st.forward, m0, x) == "BAD_STATE"              # F again in the same iteration
    st.backward_input(m1, dy)
    st.backward_weight(m1)
    st.optimizer_step()
    st.forward(m0, x)                                           # new iteration: allowed again
    assert [r[1] for r in st.log] == [0, 1, 0, 2, 1, 2, 3, 0]
    assert [r[5] for r in st.log] == [0, 0, 0, 0, 0, 0, 0, 1]


def test_tiny_op_log_golden():
    """Op log of the tiny workload equals the fixture written from its schedule."""
    import os
    cfg = get_config("tiny")
    r = oracle.run_oplist(cfg)
    path = os.path.join(os.path.dirname(__file__), "golden", "tiny_oplog.txt")
    rows = [tuple(int(v) for v in line.split()) for line in open(path)
            if line.strip() and not line.startswith("#")]
    assert [tuple(rec) for rec in r.stage.log] == rows


# ---------------------------------------------------------------------------
# Mathematical invariants
# ---------------------------------------------------------------------------

def test_causal_prefix_property():
    """y at positions < t does not depend on x at positions >= t (bitwise);
    with dy zero at positions >= t0 the input gradient beyond t0 is zero and
    dx / all weight gradients equal those of the length-t0 prefix."""
    cfg = small_cfg(layers=2, hidden=32, heads=2, ffn=64, seq=24)
    params = params64(cfg)
    shp = shape_of(cfg)
    x = gen_x(cfg, 3).astype(F64)
    y, _ = ost.stage_forward(x, params, shp)
    x2 = x.copy()
    x2[:, 10:] += np.random.default_rng(1).standard_normal(x2[:, 10:].shape)
    y2, _ = ost.stage_forward(x2, params, shp)
    assert np.array_equal(y[:, :10], y2[:, :10])
    t0 = 9
    dy = gen_dy(cfg, 3, keep_prefix=t0).astype(F64)
    _, dx, grads = decoupled(cfg, params, x, dy)
    yp, dxp, gp = decoupled(cfg, params, np.ascontiguousarray(x[:, :t0]),
                            np.ascontiguousarray(dy[:, :t0]))
    assert rel_l2(y[:, :t0], yp) < 1e-14   # different BLAS blocking at another size
    assert np.all(dx[:, t0:] == 0.0)
    assert rel_l2(dx[:, :t0], dxp) < 1e-12
    for l in range(cfg.layers):
        for p in range(12):
            assert rel_l2(grads[l][p], gp[l][p]) < 1e-12


def test_microbatch_split_invariance():
    cfg = small_cfg(micro_batch=2)
    params = params64(cfg)
    x = gen_x(cfg, 4).astype(F64)
    dy = gen_dy(cfg, 4).astype(F64)
    y, dx, g = decoupled(cfg, params, x, dy)
    parts = [decoupled(cfg, params, x[i:i + 1], dy[i:i + 1]) for i in range(2)]
    for i in range(2):
        assert rel_l2(y[i:i + 1], parts[i][0]) < 1e-14
        assert rel_l2(dx[i:i + 1], parts[i][1]) < 1e-12
    for l in range(cfg.layers):
        for p in range(12):
            assert rel_l2(g[l][p], parts[0][2][l][p] + parts[1][2][l][p]) < 1e-12


def test_linearity_in_dy():
    cfg = small_cfg()
    params = params64(cfg)
    x = gen_x(cfg, 5).astype(F64)
    d1 = gen_dy(cfg, 5).astype(F64)
    d2 = gen_dy(cfg, 6).astype(F64)
    _, dxa, ga = decoupled(cfg, params, x, 2.0 * d1 - 3.0 * d2)
    _, dx1, g1 = decoupled(cfg, params, x, d1)
    _, dx2, g2 = decoupled(cfg, params, x, d2)
    assert rel_l2(dxa, 2 * dx1 - 3 * dx2) < 1e-12
    for l in range(cfg.layers):
        for p in range(12):
            assert rel_l2(ga[l][p], 2 * g1[l][p] - 3 * g2[l][p]) < 1e-11
    _, dx0, g0 = decoupled(cfg, params, x, np.zeros_like(d1))
    assert not dx0.any() and not any(t.any() for layer in g0 for t in layer)


def test_s1_reduces_to_mlp_with_ln():
    """With one position, softmax over one key is 1 and attention returns V."""
    cfg = small_cfg(seq=1, layers=1, hidden=16, heads=4, ffn=32)
    params = params64(cfg)[0]
    x = gen_x(cfg, 7).astype(F64)
    y, _ = ost.layer_forward(x, params, shape_of(cfg))
    g1, be1, wqkv, bqkv, wo, bo, g2, be2, w1, b1, w2, b2 = params
    h = cfg.hidden

    def ln(z, g, b):
        mu = z.mean(-1, keepdims=True)
        sd = z.std(-1, keepdims=True)          # population std (ddof=0)
        return (z - mu) / np.sqrt(sd ** 2 + cfg.ln_eps) * g + b

    vproj = ln(x, g1, be1) @ wqkv[:, 2 * h:] + bqkv[2 * h:]
    H = x + vproj @ wo + bo
    from scipy.special import erf  # noqa: F401  (scipy present; tanh form below)
    u = ln(H, g2, be2) @ w1 + b1
    gel = 0.5 * u * (1 + np.tanh(np.sqrt(2 / np.pi) * (u + 0.044715 * u ** 3)))
    assert rel_l2(y, H + gel @ w2 + b2) < 1e-13


def test_layernorm_and_softmax_backward_invariants():
    rng = np.random.default_rng(3)
    z = rng.standard_normal((7, 33))
    g = 1 + 0.1 * rng.standard_normal(33)
    out, zhat, r = ost.layer_norm(z, g, np.zeros(33), 1e-5)
    assert np.allclose(zhat.mean(-1), 0, atol=1e-14)
    assert np.allclose((zhat ** 2).mean(-1), 1 / (1 + 1e-5 * r[:, 0] ** 2), rtol=1e-12)
    dout = rng.standard_normal((7, 33))
    dz = ost.layer_norm_grad_input(dout, zhat, r, g)
    assert np.allclose(dz.sum(-1), 0, atol=1e-12)
    # dz . zhat = r * sum(dout*g*zhat) * (1 - mean(zhat^2)) = r^3 * eps * sum(dout*g*zhat)
    expect = r[:, 0] ** 3 * 1e-5 * (dout * g * zhat).sum(-1)
    assert np.allclose((dz * zhat).sum(-1), expect, rtol=1e-9, atol=1e-15)
    _, zhat0, r0 = ost.layer_norm(z, g, np.zeros(33), 0.0)
    dz0 = ost.layer_norm_grad_input(dout, zhat0, r0, g)
    assert np.allclose((dz0 * zhat0).sum(-1), 0, atol=1e-12)
    q, k, v = (rng.standard_normal((1, 2, 9, 4)) for _ in range(3))
    o, p = ost.attention(q, k, v, causal=True)
    assert np.allclose(p.sum(-1), 1, atol=1e-14)
    assert np.all(p[..., np.triu_indices(9, 1)[0], np.triu_indices(9, 1)[1]] == 0)
    do = rng.standard_normal(o.shape)
    dp = np.matmul(do, np.swapaxes(v, -1, -2))
    ds = p * (dp - (dp * p).sum(-1, keepdims=True))
    assert np.allclose(ds.sum(-1), 0, atol=1e-12)


def test_gelu_against_torch_and_fd():
    torch = pytest.importorskip("torch")
    u = np.linspace(-8, 8, 2001)
    ref = torch.nn.functional.gelu(torch.tensor(u, dtype=torch.float64), approximate="tanh").numpy()
    assert np.max(np.abs(ost.gelu(u) - ref)) < 1e-14
    assert ost.gelu(np.array([0.0]))[0] == 0.0
    h = 1e-6
    fd = (ost.gelu(u + h) - ost.gelu(u - h)) / (2 * h)
    assert np.max(np.abs(ost.gelu_prime(u) - fd)) < 1e-8


# ---------------------------------------------------------------------------
# AdamW
# ---------------------------------------------------------------------------

def test_adamw_closed_form_t1():
    rng = np.random.default_rng(0)
    hp = ost.AdamHP()
    p = rng.standard_normal(1000) * 0.02
    g = rng.standard_normal(1000) * 1e-3
    p1, m1, v1 = ost.adamw_update(p, g, np.zeros_like(p), np.zeros_like(p), 1, hp, decay=True)
    assert np.allclose(p1 - p, -hp.lr * g / (np.abs(g) + hp.eps) - hp.lr * hp.weight_decay * p,
                       rtol=1e-12, atol=1e-18)
    assert np.allclose(m1, 0.1 * g, rtol=1e-15) and np.allclose(v1, 0.05 * g * g, rtol=1e-14)
    p1n, _, _ = ost.adamw_update(p, g, np.zeros_like(p), np.zeros_like(p), 1, hp, decay=False)
    assert np.allclose(p1n - p, -hp.lr * g / (np.abs(g) + hp.eps), rtol=1e-12, atol=1e-18)


def test_adamw_against_torch_optim():
    torch = pytest.importorskip("torch")
    hp = ost.AdamHP()
    rng = np.random.default_rng(1)
    p0 = rng.standard_normal(257) * 0.02
    tp = torch.nn.Parameter(torch.tensor(p0, dtype=torch.float64))
    opt = torch.optim.AdamW([tp], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay)
    p, m, v = p0.copy(), np.zeros_like(p0), np.zeros_like(p0)
    for t in range(1, 6):
        g = rng.standard_normal(257) * 10.0 ** (-t)
        tp.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        p, m, v = ost.adamw_update(p, g, m, v, t, hp, decay=True)
        assert np.allclose(p, tp.detach().numpy(), rtol=1e-13, atol=1e-18)


def test_stage_step_uses_decay_only_on_matrices():
    cfg = small_cfg(layers=1)
    st = oracle.OracleStage(cfg, gen_params(cfg))
    p_before = [t.copy() for t in st.params[0]]
    st.optimizer_step()  # no micro-batches: zero gradient, pure decay on matrices
    for pid in range(12):
        expect = p_before[pid] * (1 - 1e-4 * 0.1) if pid in ost.MATRIX_IDS else p_before[pid]
        assert np.allclose(st.params[0][pid], expect, rtol=1e-15, atol=0)


# ---------------------------------------------------------------------------
# Post-step validation, skip and rollback (section 5)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("decay", [True, False])
def test_adamw_rollback_inverts_the_step(decay):
    """Round trip at several step numbers: rollback(step(p, m, v)) == (p, m, v)."""
    rng = np.random.default_rng(7)
    hp = ost.AdamHP()
    for t in (1, 2, 7, 40):
        p = rng.standard_normal(500) * 0.02
        m = rng.standard_normal(500) * 1e-3 if t > 1 else np.zeros(500)
        v = rng.random(500) * 1e-6 if t > 1 else np.zeros(500)
        g = rng.standard_normal(500) * 1e-3
        p1, m1, v1 = ost.adamw_update(p, g, m, v, t, hp, decay=decay)
        p0, m0, v0 = ost.adamw_rollback(p1, g, m1, v1, t, hp, decay=decay)
        assert rel_l2(p0, p) < 1e-12
        assert np.abs(m0 - m).max() <= 1e-12 * max(np.abs(g).max(), np.abs(m).max())
        assert np.abs(v0 - v).max() <= 1e-12 * max((g * g).max(), np.abs(v).max())
        # undoing step t with the bias correction of another step number is not an inverse
        pw, _, _ = ost.adamw_rollback(p1, g, m1, v1, t + 1, hp, decay=decay)
        assert rel_l2(pw, p) > 1e-6


def test_adamw_rollback_against_torch_optim_history():
    """Two torch AdamW steps then one rollback land on torch's one-step state."""
    torch = pytest.importorskip("torch")
    hp = ost.AdamHP()
    rng = np.random.default_rng(3)
    p0 = rng.standard_normal(300) * 0.02
    g1, g2 = rng.standard_normal(300) * 1e-3, rng.standard_normal(300) * 1e-3
    tp = torch.nn.Parameter(torch.tensor(p0, dtype=torch.float64))
    opt = torch.optim.AdamW([tp], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay)
    tp.grad = torch.tensor(g1, dtype=torch.float64)
    opt.step()
    after1 = tp.detach().numpy().copy()
    st = opt.state[tp]
    m_1, v_1 = st["exp_avg"].numpy().copy(), st["exp_avg_sq"].numpy().copy()
    tp.grad = torch.tensor(g2, dtype=torch.float64)
    opt.step()
    p, m, v = ost.adamw_rollback(tp.detach().numpy(), g2, st["exp_avg"].numpy(),
                                 st["exp_avg_sq"].numpy(), 2, hp, decay=True)
    assert rel_l2(p, after1) < 1e-12 and rel_l2(m, m_1) < 1e-10 and rel_l2(v, v_1) < 1e-10


def _stage_after_iteration(cfg):
    st = oracle.OracleStage(cfg, gen_params(cfg))
    for op in op_list(cfg, with_step=False):
        if op.kind == "F":
            st.forward(op.mb, gen_x(cfg, op.mb.j, op.mb.k))
        elif op.kind == "B":
            st.backward_input(op.mb, gen_dy(cfg, op.mb.j, op.mb.k))
        else:
            st.backward_weight(op.mb)
    return st


def test_stage_skip_and_rollback_rules():
    cfg = small_cfg(layers=1, n_mb=2)
    st = _stage_after_iteration(cfg)
    before = copy.deepcopy((st.params, st.m, st.v, st.t))
    st.optimizer_skip()
    assert st.t == before[3] and st.iter == 1
    for l in range(cfg.layers):
        for p in range(12):
            assert np.array_equal(st.params[l][p], before[0][l][p])
    with pytest.raises(oracle.StageError):          # nothing to undo after a skip
        st.optimizer_rollback()
    # a step, then its rollback: back to the state before the step
    st2 = _stage_after_iteration(cfg)
    st2.optimizer_step(grad_scale=0.5)
    st2.optimizer_rollback()
    assert st2.t == 0
    for l in range(cfg.layers):
        for p in range(12):
            assert rel_l2(st2.params[l][p], before[0][l][p]) < 1e-12
            assert np.abs(st2.m[l][p]).max() < 1e-15 and np.abs(st2.v[l][p]).max() < 1e-20
    with pytest.raises(oracle.StageError):          # only once
        st2.optimizer_rollback()
    # after any call that follows the step, its rollback is refused
    st3 = _stage_after_iteration(cfg)
    st3.optimizer_step()
    st3.forward(MB(0), gen_x(cfg, 0))
    with pytest.raises(oracle.StageError):
        st3.optimizer_rollback()
    assert [r[1] for r in st2.log[-2:]] == [ost.OP_STEP, ost.OP_ROLLBACK]
    assert st2.log[-1][5] == st2.log[-2][5]          # the rollback belongs to the stepped iteration


def test_grad_check_matches_fused_gradient_norm():
    """The squared norm reported equals that of the fused reverse pass's
    gradient (an independent path), and planted non-finite entries are counted."""
    cfg = small_cfg(layers=2, n_mb=2)
    st = _stage_after_iteration(cfg)
    params = params64(cfg)
    shp = shape_of(cfg)
    total = None
    for mb in (MB(0), MB(1)):
        x = gen_x(cfg, mb.j, mb.k).astype(F64)
        y, caches = ost.stage_forward(x, params, shp)
        _, g = ost.stage_backward_fused(gen_dy(cfg, mb.j, mb.k).astype(F64), caches, params)
        total = g if total is None else [[a + b for a, b in zip(la, lb)] for la, lb in zip(total, g)]
    ref = sum(float(np.sum((0.5 * t) ** 2)) for layer in total for t in layer)
    ss, bad = st.grad_check(grad_scale=0.5)
    assert bad == 0 and abs(ss - ref) <= 1e-12 * ref
    st.grads[0][2][0, 0] = np.nan
    st.grads[1][9][3] = np.inf
    ss2, bad2 = st.grad_check()
    assert bad2 == 2 and np.isfinite(ss2)
    fresh = oracle.OracleStage(cfg, gen_params(cfg))
    assert fresh.grad_check() == (0.0, 0)


# ---------------------------------------------------------------------------
# Mutation checks: a planted mistake in the oracle must fail a pin
# ---------------------------------------------------------------------------

def _pins_pass(cfg):
    params = params64(cfg)
    x = gen_x(cfg, 1).astype(F64)
    dy = gen_dy(cfg, 1).astype(F64)
    y, dx, grads = decoupled(cfg, params, x, dy)
    ty, tdx, tg = torch_stage(cfg, params, x, dy)
    ok = rel_l2(y, ty) < 1e-10 and rel_l2(dx, tdx) < 1e-8
    ok = ok and all(rel_l2(grads[l][p], tg[l][p]) < 1e-8 for l in range(cfg.layers) for p in range(12))
    return ok


@pytest.mark.parametrize("mutation", ["gelu_sign", "ln_drop_term", "attn_transpose", "attn_scale"])
def test_planted_mistakes_are_caught(monkeypatch, mutation):
    cfg = small_cfg(layers=1, hidden=16, heads=2, ffn=32, seq=7)
    assert _pins_pass(cfg)
    if mutation == "gelu_sign":
        orig = ost.gelu_prime
        monkeypatch.setattr(ost, "gelu_prime", lambda u: orig(-u))
    elif mutation == "ln_drop_term":
        def bad(dout, zhat, rstd, g):
            dz = dout * g
            return rstd * (dz - dz.mean(-1, keepdims=True))
        monkeypatch.setattr(ost, "layer_norm_grad_input", bad)
    elif mutation == "attn_transpose":
        orig = ost.attention_grad

        def bad(do, q, k, v, p):
            dq, dk, dv = orig(do, q, k, v, p)
            return dk, dq, dv
        monkeypatch.setattr(ost, "attention_grad", bad)
    elif mutation == "attn_scale":
        orig = ost.attention

        def bad(q, k, v, causal):
            return orig(q * 2.0, k, v, causal)
        monkeypatch.setattr(ost, "attention", bad)
    assert not _pins_pass(cfg)
