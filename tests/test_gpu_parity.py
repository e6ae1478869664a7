"""Parity of the HIP stage (through the C ABI) with the fp64 oracle.

Bars (rel-L2 = ||gpu - oracle|| / ||oracle|| per tensor, fp64 on the host):
  fp32 stages  <= 1e-5;  bf16 stages (bf16 storage, fp32 accumulate) <= 2e-2;
  op logs identical.
Small ragged workloads are compared element by element on every output.
The full-size workloads are compared on what the oracle can afford at full
size, using causality (a property that holds at any size): y at the first t0
positions depends only on x[:t0]; and with dy zero beyond t0, dx and every
weight gradient equal those of the length-t0 prefix.  The GPU always runs the
full sequence length, i.e. the launch configuration the benchmark times.
"""
import functools

import numpy as np
import pytest

import oracle
from synth import CONFIGS, TEST_CONFIGS, MB, gen_dy, gen_params, gen_x, get_config, op_list
from tests.conftest import compare_grads, rel_l2
from tests.gpu_harness import log, run_gpu

pytestmark = pytest.mark.gpu

MATRIX = (2, 4, 8, 10)


def tol(cfg):
    return 1e-5 if cfg.dtype == "f32" else 2e-2


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    import paper_2405_14009_amd  # noqa: F401  (fails loudly if the library is missing)
    yield
    torch.cuda.empty_cache()


def compare_state(cfg, g, o, t, zero_init=()):
    """grads after the last W, then params / m / v after the step.

    The K block of the QKV bias has an exactly zero gradient (adding a
    constant to every key of a query leaves its softmax unchanged), so both
    sides hold rounding noise there and the first AdamW update is the sign of
    that noise: its parameters are not compared; instead its gradient must be
    negligible next to the V block's."""
    worst = {}
    h = cfg.hidden
    for l in range(cfg.layers):
        for p in range(12):
            worst[("grad", l, p)] = rel_l2(g.grads[l][p], o.grads[l][p])
            worst[("m", l, p)] = rel_l2(g.m[l][p], o.stage.m[l][p])
            worst[("v", l, p)] = rel_l2(g.v[l][p], o.stage.v[l][p])
            if (l, p) in zero_init:
                continue
            if p == 3:
                keep = np.r_[0:h, 2 * h:3 * h]
                worst[("param", l, p)] = rel_l2(g.params[l][p][keep], o.stage.params[l][p][keep])
                ratio = np.linalg.norm(g.grads[l][p][h:2 * h]) / np.linalg.norm(g.grads[l][p][2 * h:])
                log(f"  layer {l}: |grad b_k| / |grad b_v| = {ratio:.2e}")
                assert ratio < (1e-4 if cfg.dtype == "f32" else 2e-2)
            else:
                worst[("param", l, p)] = rel_l2(g.params[l][p], o.stage.params[l][p])
    bad = {k: v for k, v in worst.items() if v > t}
    assert not bad, bad
    return max(worst.values())


def check_adam_on_gpu_grads(cfg, g, params0, hp=None):
    """The optimizer alone: the oracle's AdamW applied to the GPU's own
    gradients reproduces the GPU's params / m / v (first step)."""
    hp = hp or oracle.AdamHP()
    for l in range(cfg.layers):
        for p in range(12):
            P, M, V = oracle.adamw_update(params0[l][p].astype(np.float64), g.grads[l][p].astype(np.float64),
                                          0.0, 0.0, 1, hp, decay=p in MATRIX)
            assert rel_l2(g.params[l][p], P) < 1e-6, (l, p)
            assert rel_l2(g.m[l][p], M) < 1e-6 and rel_l2(g.v[l][p], V) < 1e-5, (l, p)


@pytest.mark.parametrize("name", ["tiny", "tiny_noncausal", "tiny_perturbed", "small_f32", "small_bf16",
                                  "wide_bf16", "persist_bf16"])
def test_elementwise_parity(name):
    cfg = get_config(name)
    if name == "persist_bf16":
        # FC1 / FC2 weight gradients: 320 tiles of 256 x 256 (ragged), a multiple of 8 and more
        # than one per compute unit, so the launcher takes the persistent kernel
        import torch
        cus = torch.cuda.get_device_properties(0).multi_processor_count
        tiles = -(-cfg.hidden // 256) * -(-cfg.ffn // 256)
        assert tiles % 8 == 0 and tiles > cus, (tiles, cus)
    log(f"[parity] {name}: shapes L={cfg.layers} h={cfg.hidden} a={cfg.heads} f={cfg.ffn} "
        f"s={cfg.seq} b={cfg.micro_batch} {cfg.dtype} causal={cfg.causal}")
    g = run_gpu(cfg)
    o = oracle.run_oplist(cfg)
    t = tol(cfg)
    assert g.log == [tuple(r) for r in o.stage.log]
    for mb in o.y:
        assert rel_l2(g.y[mb], o.y[mb]) < t, ("y", mb, rel_l2(g.y[mb], o.y[mb]))
        assert rel_l2(g.dx[mb], o.dx[mb]) < t, ("dx", mb, rel_l2(g.dx[mb], o.dx[mb]))
    zero_init = {(l, p) for l in range(cfg.layers) for p in (1, 3, 5, 7, 9, 11)} if not cfg.perturbed else set()
    worst = compare_state(cfg, g, o, t, zero_init if cfg.dtype == "bf16" else ())
    check_adam_on_gpu_grads(cfg, g, gen_params(cfg))
    log(f"[parity] {name}: worst state rel-L2 {worst:.2e}")


@pytest.mark.parametrize("variant", [
    dict(causal=False),
    dict(seq=328),                                    # ragged: last query / key blocks partial
    dict(seq=328, causal=False, micro_batch=3, n_mb=2),
    dict(seq=64, micro_batch=3, n_mb=2),              # one key block
    dict(seq=1000, n_mb=2),                           # 8 query blocks: 4 pairs of unequal halves
    dict(seq=136, n_mb=2),                            # 2 query blocks, the last one's key range capped at s
    dict(seq=8, micro_batch=4, n_mb=2),               # the shortest sequence the stage takes
])
def test_attention_variants_parity(variant):
    """bf16 stages with head dimension 128 take the fused attention path
    (scores never materialised); non-causal, ragged and multi-sequence
    micro-batches against the oracle."""
    cfg = get_config("small_bf16").with_(**variant)
    log(f"[attn] {variant}: s={cfg.seq} b={cfg.micro_batch} causal={cfg.causal}")
    g = run_gpu(cfg)
    o = oracle.run_oplist(cfg)
    t = tol(cfg)
    assert g.log == [tuple(r) for r in o.stage.log]
    for mb in o.y:
        assert rel_l2(g.y[mb], o.y[mb]) < t, ("y", mb, rel_l2(g.y[mb], o.y[mb]))
        assert rel_l2(g.dx[mb], o.dx[mb]) < t, ("dx", mb, rel_l2(g.dx[mb], o.dx[mb]))
    zero_init = {(l, p) for l in range(cfg.layers) for p in (1, 3, 5, 7, 9, 11)} if not cfg.perturbed else set()
    worst = compare_state(cfg, g, o, t, zero_init)
    log(f"[attn] {variant}: worst state rel-L2 {worst:.2e}")


@pytest.mark.parametrize("seq", [1024, 1000])
def test_causal_block_attention_parity(seq):
    """Causal attention through the per-query-block kernels (the path of the
    40-head 13B stage): the grid of query-block pairs would fill its last
    round of compute units poorly, so each block of 128 queries is one
    workgroup walking its own causal key range (2 .. 16 key blocks of 64,
    with the online softmax rescaled across them).  Every output, and every
    128-query block of y and dx on its own, against the oracle."""
    from paper_2405_14009_amd import Stage
    cfg = get_config("block_bf16").with_(seq=seq)
    stage = Stage.from_config(cfg)
    path = stage.attention_kernels()
    log(f"[block attn] s={seq} b={cfg.micro_batch} heads={cfg.heads}: {path} kernels")
    assert path == "block"
    params = gen_params(cfg)
    stage.load_params(params)
    g = run_gpu(cfg, stage=stage)
    stage.close()
    o = oracle.run_oplist(cfg, params=params)
    t = tol(cfg)
    assert g.log == [tuple(r) for r in o.stage.log]
    worst = 0.0
    for mb in o.y:
        for name, a, b in (("y", g.y[mb], o.y[mb]), ("dx", g.dx[mb], o.dx[mb])):
            assert rel_l2(a, b) < t, (name, mb, rel_l2(a, b))
            for sq in range(cfg.micro_batch):
                for r0 in range(0, cfg.seq, 128):
                    e = rel_l2(a[sq, r0:r0 + 128], b[sq, r0:r0 + 128])
                    worst = max(worst, e)
                    assert e < t, (name, mb, sq, r0, e)
    log(f"[block attn] s={seq}: worst per-block rel-L2 of y, dx {worst:.2e}")
    worst = compare_state(cfg, g, o, t)
    check_adam_on_gpu_grads(cfg, g, params)
    log(f"[block attn] s={seq}: worst state rel-L2 {worst:.2e}")


def test_w_order_and_determinism():
    """Deferred W in another order gives the same gradients (fp32 sums in a
    different order: rel <= 1e-6); the same order is bitwise reproducible."""
    cfg = get_config("small_bf16")
    ops = op_list(cfg, with_step=False)
    fwd = [o for o in ops if o.kind != "W"]
    ws = [o for o in ops if o.kind == "W"]
    a = run_gpu(cfg, fwd + ws, keep_outputs=False)
    b = run_gpu(cfg, fwd + ws, keep_outputs=False)
    c = run_gpu(cfg, fwd + ws[::-1], keep_outputs=False)
    for l in range(cfg.layers):
        for p in range(12):
            assert np.array_equal(a.grads[l][p], b.grads[l][p]), (l, p)
            assert rel_l2(c.grads[l][p], a.grads[l][p]) < 1e-6, (l, p)


def _grouped(ops):
    from synth.schedules import Op
    out = []
    for op in ops:
        if op.kind == "W" and out and out[-1].kind == "W*":
            out[-1].mb.append(op.mb)
        elif op.kind == "W":
            out.append(Op("W*", [op.mb]))
        else:
            out.append(op)
    return out


@pytest.mark.parametrize("name,seq", [("small_bf16", None), ("small_bf16", 328), ("small_f32", None),
                                      ("persist_bf16", None)])
def test_batched_weight_pass(name, seq):
    """One weight pass over several deferred micro-batches (one product per
    parameter over their concatenated tokens; for bf16 token counts that are
    not a multiple of 64, one product per micro-batch) equals one call per
    micro-batch (fp32 sums in another order: rel <= 1e-6), logs the same
    records, and matches the oracle."""
    cfg = get_config(name)
    if seq:
        cfg = cfg.with_(seq=seq)
    log(f"[batched W] {name} s={cfg.seq} b={cfg.micro_batch} T={cfg.seq * cfg.micro_batch} {cfg.dtype}")
    ops = op_list(cfg, with_step=False)
    fwd = [o for o in ops if o.kind != "W"]
    ws = [o for o in ops if o.kind == "W"]
    from synth.schedules import Op
    a = run_gpu(cfg, fwd + ws, keep_outputs=False)
    b = run_gpu(cfg, fwd + [Op("W*", [o.mb for o in ws])], keep_outputs=False)
    c = run_gpu(cfg, _grouped(ops) + [Op("STEP")], keep_outputs=False)
    assert a.log == b.log
    for l in range(cfg.layers):
        for p in range(12):
            assert rel_l2(b.grads[l][p], a.grads[l][p]) < 1e-6, (l, p)
    o = oracle.run_oplist(cfg)
    assert c.log == [tuple(r) for r in o.stage.log]
    zero_init = {(l, p) for l in range(cfg.layers) for p in (1, 3, 5, 7, 9, 11)} if not cfg.perturbed else set()
    compare_state(cfg, c, o, tol(cfg), zero_init if cfg.dtype == "bf16" else ())


def test_peer_reroute_invariance_on_gpu():
    """Two peers of one stage on one GPU; the failed pipeline's micro-batches
    are re-routed round-robin; the peers' gradient sum equals the fault-free
    sum, and each micro-batch's outputs match whoever runs it."""
    cfg = get_config("small_f32").with_(n_mb=2, layers=1, schedule="coupled")
    from synth.schedules import Op
    dp = 3
    work = {k: [MB(j, k) for j in range(cfg.n_mb)] for k in range(dp)}

    def run(assign):
        tot, outs = None, {}
        for ks, mbs in assign.items():
            ops = [Op(kind, m) for m in mbs for kind in ("F", "B", "W")]
            r = run_gpu(cfg.with_(max_stashed_mb=len(mbs), max_inflight_mb=len(mbs)), ops,
                        pipeline_id=ks)
            outs.update({("y",) + k: v for k, v in r.y.items()})
            g = [np.concatenate([t.ravel() for t in layer]) for layer in r.grads]
            tot = g if tot is None else [x + y for x, y in zip(tot, g)]
        return tot, outs

    ff, ff_out = run(work)
    assign = {0: list(work[0]), 2: list(work[2])}
    for i, m in enumerate(work[1]):
        assign[[0, 2][i % 2]].append(m)
    rr, rr_out = run(assign)
    for k in ff_out:
        assert np.array_equal(ff_out[k], rr_out[k])
    for x, y in zip(rr, ff):
        assert rel_l2(x, y) < 1e-6


def test_staggered_two_stages():
    """Stage i steps while stage i+1 (another handle on the same GPU) still
    has deferred W pending; both end equal to their own oracle runs."""
    cfg = get_config("small_f32").with_(layers=1)
    ops = op_list(cfg)
    step = ops[-1]
    body = ops[:-1]
    from paper_2405_14009_amd import Stage
    s0 = Stage.from_config(cfg, stage_index=0)
    s1 = Stage.from_config(cfg, stage_index=1)
    p0 = gen_params(cfg)
    p1 = gen_params(cfg.with_(seed=1))
    s0.load_params(p0)
    s1.load_params(p1)
    nw = sum(o.kind == "W" for o in body)
    # stage 1 runs everything but its last two W; stage 0 finishes and steps.
    run_gpu(cfg, [o for o in body], stage=s0, read_state=False, keep_outputs=False)
    w1 = [o for o in body if o.kind == "W"]
    run_gpu(cfg, [o for o in body if o.kind != "W"] + w1[:nw - 2], stage=s1, read_state=False,
            keep_outputs=False)
    s0.optimizer_step()
    r1 = run_gpu(cfg, w1[nw - 2:] + [step], stage=s1)
    r0 = run_gpu(cfg, [], stage=s0)
    o0 = oracle.run_oplist(cfg, params=p0)
    o1 = oracle.run_oplist(cfg, params=p1)
    for r, o in ((r0, o0), (r1, o1)):
        compare_state(cfg, r, o, 1e-5)
    s0.close()
    s1.close()


# ---------------------------------------------------------------------------
# Full-size workloads: causal-prefix sampling
# ---------------------------------------------------------------------------

T0 = 64


@functools.lru_cache(maxsize=None)
def full_params(name):
    """Seeded parameters of a full-size workload, generated once per session
    (tens of seconds for the larger stages); callers must not modify them."""
    return gen_params(CONFIGS[name])


@pytest.mark.parametrize("name", ["gpt1.3b", "gpt6.7b", "gpt13b", "gpt175b"])
def test_fullsize_prefix_parity(name):
    _fullsize(name, batched=False)


@pytest.mark.parametrize("name", ["gpt6.7b", "gpt13b"])
def test_fullsize_batched_weight_pass(name):
    """The launch configuration the benchmark times: consecutive deferred weight
    passes of the op list run as one batched call (16 micro-batches, a
    32768-token segmented reduction, for the 6.7B stage)."""
    _fullsize(name, batched=True)


def _fullsize(name, batched):
    cfg = CONFIGS[name]
    log(f"[fullsize] {name}: L={cfg.layers} h={cfg.hidden} a={cfg.heads} f={cfg.ffn} "
        f"s={cfg.seq} b={cfg.micro_batch} n_mb={cfg.n_mb}, prefix t0={T0}")
    params = full_params(name)
    ops = op_list(cfg)
    # 1) real inputs: y[:, :t0] against the oracle forward of the prefix
    pre = cfg.with_(seq=T0)
    ps = [[p.astype(np.float64) for p in layer] for layer in params]
    shp = oracle.LayerShape(cfg.heads, cfg.causal, cfg.ln_eps)
    g = run_gpu(cfg, [o for o in ops if o.kind == "F"][:1], params=params, read_state=False,
                max_stashed_mb=1, max_inflight_mb=1)
    for mb in g.y:
        yo, _ = oracle.stage_forward(gen_x(cfg, mb[0], mb[1], seq=T0).astype(np.float64), ps, shp)
        e = rel_l2(g.y[mb][:, :T0], yo)
        log(f"[fullsize] {name}: y prefix rel-L2 {e:.2e}")
        assert e < 2e-2
    del g
    # 2) dy zero beyond t0: full op list on the GPU, prefix op list on the oracle
    dy_fn = lambda j, k: gen_dy(cfg, j, k, keep_prefix=T0)
    g = run_gpu(cfg, _grouped(ops) if batched else ops, params=params, dy_fn=dy_fn)
    o = oracle.run_oplist(pre, ops, params=params,
                          x_fn=lambda j, k: gen_x(cfg, j, k, seq=T0),
                          dy_fn=lambda j, k: gen_dy(cfg, j, k)[:, :T0])
    assert g.log == [tuple(r) for r in o.stage.log]
    for mb in o.dx:
        assert not np.any(g.dx[mb][:, T0:]), mb
        e = rel_l2(g.dx[mb][:, :T0], o.dx[mb])
        assert e < 2e-2, ("dx", mb, e)
    zero_init = {(l, p) for l in range(cfg.layers) for p in (1, 3, 5, 7, 9, 11)}
    worst = compare_state(cfg, g, o, 2e-2, zero_init)
    check_adam_on_gpu_grads(cfg, g, params)
    log(f"[fullsize] {name}: worst state rel-L2 {worst:.2e}")



@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["gpt1.3b", "gpt6.7b", "gpt13b", "gpt175b"])
def test_fullsize_full_sequence_first_microbatch(name):
    """The first micro-batch of each full-size op list at its full sequence
    length, on its own seeded x and dy: F, B_input and B_weight on the GPU
    (the launch configuration the benchmark times) against the fp64 oracle
    of the whole sequence; y, dx and every gradient."""
    import time
    from paper_2405_14009_amd import RC_READ_GRAD, Stage
    from synth.schedules import Op
    cfg = CONFIGS[name]
    mb = next(o.mb for o in op_list(cfg) if o.kind == "F")
    log(f"[full seq] {name}: micro-batch {tuple(mb)}, L={cfg.layers} h={cfg.hidden} s={cfg.seq} "
        f"b={cfg.micro_batch}")
    params = full_params(name)
    stage = Stage.from_config(cfg, max_stashed_mb=1, max_inflight_mb=1)
    log(f"[full seq] {name}: attention kernels {stage.attention_kernels()}")
    stage.load_params(params)
    g = run_gpu(cfg, [Op("F", mb), Op("B", mb), Op("W", mb)], stage=stage, read_state=False)
    grads = stage.read_all(RC_READ_GRAD)
    stage.close()
    del stage
    t0 = time.perf_counter()
    shp = oracle.LayerShape(cfg.heads, cfg.causal, cfg.ln_eps)
    ps = [[p.astype(np.float64) for p in layer] for layer in params]
    yo, caches = oracle.stage_forward(gen_x(cfg, mb.j, mb.k).astype(np.float64), ps, shp)
    dxo, stashes = oracle.stage_backward_input(gen_dy(cfg, mb.j, mb.k).astype(np.float64), caches, ps)
    del caches, ps
    go = oracle.stage_backward_weight(stashes)
    del stashes
    log(f"[full seq] {name}: oracle {time.perf_counter() - t0:.1f} s")
    ey, edx = rel_l2(g.y[tuple(mb)], yo), rel_l2(g.dx[tuple(mb)], dxo)
    eg = compare_grads(cfg, grads, go, 2e-2)
    log(f"[full seq] {name}: rel-L2 y {ey:.2e}, dx {edx:.2e}, worst gradient {eg:.2e}")
    assert ey < 2e-2 and edx < 2e-2, (ey, edx)
