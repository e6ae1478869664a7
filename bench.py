#!/usr/bin/env python3
"""Benchmark one pipeline stage's decoupled-backprop training iteration on one MI355X.

A step is one iteration of the stage's op list: every micro-batch's forward
(F), input-gradient pass (B_input) and deferred weight-gradient pass
(B_weight), then the stage's own AdamW step, on seeded synthetic inputs that
are resident in HBM before the timed region.  The default workload is the
GPT-6.7B-shaped stage (4 pre-LN layers, hidden 4096, 32 heads, FFN 16384,
causal sequence 2048, micro-batch 1, 16 micro-batches with all weight passes
deferred and issued in a shuffled order).

Prints one JSON line: stage TFLOP/s (value), micro-batches/s, F/B/W TFLOP/s,
GEMM-class TFLOP/s and their fraction of the bf16 MFMA peak, the roofline of
the dominant kernel class, and the fp64 CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA (published)
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
# Dense bf16 MFMA peak per GHz of shader clock: 256 CUs x 4 SIMDs x 1024 flop/clk
# (2516.6 TFLOP/s at the nominal 2.4 GHz, published as 2.5 PFLOP/s).
PEAK_PER_GHZ = 256 * 4 * 1024 / 1e3
METRIC = "stage F/B/W TFLOP/s + % bf16 MFMA peak; micro-batches/sec per stage"


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def workload_name(cfg) -> str:
    return (f"{cfg.name}-stage: {cfg.layers} pre-LN layers, hidden {cfg.hidden}, {cfg.heads} heads, "
            f"ffn {cfg.ffn}, {'causal ' if cfg.causal else ''}seq {cfg.seq}, micro-batch "
            f"{cfg.micro_batch}, {cfg.n_mb} micro-batches ({len(cfg.rerouted)} re-routed), "
            f"schedule {cfg.schedule}, {cfg.dtype}")


def cpu_baseline(cfg, params) -> dict:
    """The fp64 oracle (as it stands) on a bounded sample of the workload:
    F + B_input + B_weight of one layer at full shape, for successive
    micro-batches until at least 10 s of CPU work have run."""
    import numpy as np
    import oracle
    from synth import gen_dy, gen_x
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    P = [p.astype(np.float64) for p in params[0]]
    shp = oracle.LayerShape(cfg.heads, cfg.causal, cfg.ln_eps)
    t = {"F": 0.0, "B": 0.0, "W": 0.0}
    n = 0
    while sum(t.values()) < 10.0 and n < cfg.n_mb:
        x = gen_x(cfg, n).astype(np.float64)
        dy = gen_dy(cfg, n).astype(np.float64)
        t0 = time.perf_counter()
        y, cache = oracle.layer_forward(x, P, shp)
        t1 = time.perf_counter()
        dx, ws = oracle.layer_backward_input(dy, cache, P)
        t2 = time.perf_counter()
        oracle.layer_backward_weight(ws)
        t3 = time.perf_counter()
        t["F"] += t1 - t0
        t["B"] += t2 - t1
        t["W"] += t3 - t2
        n += 1
    F, B, W = cfg.flops_per_layer()
    flops = n * (F + B + W)
    dt = sum(t.values())
    return {"value": round(flops / dt / 1e12, 4), "unit": "TFLOP/s", "cores": int(cores),
            "kind": "oracle",
            "pass_tflops": {k: round(n * fl / t[k] / 1e12, 4) for k, fl in (("F", F), ("B", B), ("W", W))},
            "sample": (f"fp64 numpy oracle: F + B_input + B_weight of 1 of {cfg.layers} layers for {n} of "
                       f"{cfg.n_mb} micro-batches at full shape ({flops / 1e9:.0f} GFLOP algorithmic) "
                       f"in {dt:.1f} s")}


def cpu_baseline_all() -> dict:
    """The fp64 oracle per workload: F, B_input and B_weight of one
    micro-batch through all of the stage's layers (the first micro-batch of
    its op list, full shape), and for the tiny workload its whole op list
    (every micro-batch and the AdamW step).  Minutes of CPU time; not part of
    the default run."""
    import numpy as np
    import oracle
    from synth import CONFIGS, gen_dy, gen_params, gen_x, op_list
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    out = {"cores": int(cores), "kind": "oracle", "workloads": {}}
    for name, cfg in CONFIGS.items():
        mb = next(o.mb for o in op_list(cfg) if o.kind == "F")
        ps = [[p.astype(np.float64) for p in layer] for layer in gen_params(cfg)]
        shp = oracle.LayerShape(cfg.heads, cfg.causal, cfg.ln_eps)
        x = gen_x(cfg, mb.j, mb.k).astype(np.float64)
        dy = gen_dy(cfg, mb.j, mb.k).astype(np.float64)
        t0 = time.perf_counter()
        y, caches = oracle.stage_forward(x, ps, shp)
        t1 = time.perf_counter()
        dx, stashes = oracle.stage_backward_input(dy, caches, ps)
        t2 = time.perf_counter()
        del caches
        oracle.stage_backward_weight(stashes)
        t3 = time.perf_counter()
        F, B, W = (cfg.layers * f for f in cfg.flops_per_layer())
        e = {"F_s": round(t1 - t0, 3), "B_s": round(t2 - t1, 3), "W_s": round(t3 - t2, 3),
             "tflops": {"F": round(F / (t1 - t0) / 1e12, 4), "B": round(B / (t2 - t1) / 1e12, 4),
                        "W": round(W / (t3 - t2) / 1e12, 4)}}
        if name == "tiny":
            t4 = time.perf_counter()
            oracle.run_oplist(cfg)
            e["op_list_s"] = round(time.perf_counter() - t4, 3)
        out["workloads"][name] = e
        log(f"cpu baseline {name}: {e}")
        del ps, stashes
    return out


def measured_traffic(cfg, kernel_class: str):
    """HBM bytes per launch of a kernel class from the committed rocprofv3
    counter summary of this workload (FETCH_SIZE + WRITE_SIZE, copy-calibrated),
    or None when there is none or the kernel sources changed since."""
    path = os.path.join(ROOT, "profiles", f"stage_{cfg.name}_kernels.md")
    if not os.path.exists(path):
        return None, "no counter summary for this workload"
    txt = open(path).read()
    try:
        block = json.loads(txt.split("```json", 1)[1].split("```", 1)[0])
    except (IndexError, ValueError):
        return None, "counter summary unreadable"
    from paper_2405_14009_amd.profile_summary import sources_digest
    if block.get("sources_sha256") != sources_digest():
        return None, "kernels changed since the counters were taken"
    e = block.get("classes", {}).get(kernel_class, {})
    if "bytes_per_dispatch" not in e:
        return None, "no counter reading for this kernel class"
    return e["bytes_per_dispatch"], os.path.relpath(path, ROOT)


def profile_clocks(cfg) -> dict:
    """Sustained shader clock (GHz) per kernel class from the committed
    rocprofv3 counter summary of this workload (GRBM_GUI_ACTIVE over the
    dispatch time), or {} when there is none or the kernel sources changed."""
    path = os.path.join(ROOT, "profiles", f"stage_{cfg.name}_kernels.md")
    if not os.path.exists(path):
        return {}
    try:
        block = json.loads(open(path).read().split("```json", 1)[1].split("```", 1)[0])
    except (IndexError, ValueError):
        return {}
    from paper_2405_14009_amd.profile_summary import sources_digest
    if block.get("sources_sha256") != sources_digest():
        return {}
    out = {k: e["sclk_ghz"] for k, e in block.get("classes", {}).items() if e.get("sclk_ghz")}
    if out:
        out["_source"] = os.path.relpath(path, ROOT)
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="gpt6.7b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--single-w", action="store_true",
                    help="headline with one weight-pass call per micro-batch instead of merging "
                         "consecutive weight passes of the op list into one batched call")
    ap.add_argument("--no-single-w-leg", action="store_true",
                    help="skip the second leg that times the same op list with one weight-pass "
                         "call per micro-batch")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run three plain 1 GiB device copies (calibrates the HBM byte "
                         "counters of a profiler run) and exit")
    ap.add_argument("--no-profile", action="store_true",
                    help="skip the per-kernel events (for external profilers)")
    ap.add_argument("--cpu-baseline-all", action="store_true",
                    help="only time the fp64 oracle on one micro-batch of every workload (and the "
                         "tiny op list) and print it as JSON; no device work")
    args = ap.parse_args()
    if args.cpu_baseline_all:
        print(json.dumps(cpu_baseline_all()), flush=True)
        return 0
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one stage on one GPU; the library runs no collectives, so there "
              "is no multi-GPU run to measure (use --gpus 1)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2405_14009_amd import Stage
    from synth import get_config, gen_dy, gen_params, gen_x, op_list

    def to_device(a, dtype):
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")
        return t.to(torch.bfloat16) if dtype == "bf16" else t

    if not torch.cuda.is_available():
        print("no HIP device", file=sys.stderr)
        return 1
    if args.copy_probe:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("copied 3 x 1 GiB")
        return 0
    cfg = get_config(args.config)
    ops = op_list(cfg)
    log(f"workload {workload_name(cfg)}")
    t = time.perf_counter()
    params = gen_params(cfg)
    stage = Stage.from_config(cfg)
    stage.load_params(params)
    xs = {tuple(o.mb): to_device(gen_x(cfg, o.mb.j, o.mb.k), cfg.dtype) for o in ops if o.kind == "F"}
    dys = {tuple(o.mb): to_device(gen_dy(cfg, o.mb.j, o.mb.k), cfg.dtype) for o in ops if o.kind == "F"}
    ys = {k: torch.empty_like(v) for k, v in xs.items()}
    dxs = {k: torch.empty_like(v) for k, v in xs.items()}
    torch.cuda.synchronize()
    log(f"setup {time.perf_counter() - t:.1f} s (stage arenas "
        f"{(stage.state_bytes + stage.stash_bytes + stage.work_bytes) / 2**30:.1f} GiB)")

    # Deferred weight passes that follow each other in the op list run as one
    # batched call (same gradients and op-log records as one call each).
    def group(single):
        out = []
        for op in ops:
            if (op.kind == "W" and not single and out and out[-1][0] == "W" and len(out[-1][1]) < 32):
                out[-1][1].append(op.mb)
            else:
                out.append((op.kind, [op.mb]))
        return out

    steps_ops = group(args.single_w)

    def run_step(events=None, plan=None):
        for kind, mbs in (plan or steps_ops):
            if events is not None:
                a = torch.cuda.Event(enable_timing=True)
                a.record()
            if kind == "F":
                stage.forward(mbs[0], xs[tuple(mbs[0])], ys[tuple(mbs[0])])
            elif kind == "B":
                stage.backward_input(mbs[0], dys[tuple(mbs[0])], dxs[tuple(mbs[0])])
            elif kind == "W":
                if len(mbs) == 1:
                    stage.backward_weight(mbs[0])
                else:
                    stage.backward_weight_many(mbs)
            else:
                stage.optimizer_step()
            if events is not None:
                b = torch.cuda.Event(enable_timing=True)
                b.record()
                events.append((kind, a, b, len(mbs)))

    for i in range(args.warmup):
        run_step()
        torch.cuda.synchronize()
        log(f"warmup step {i + 1}/{args.warmup} done")

    # The headline figure: K un-instrumented steps between synchronisations.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        run_step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    log(f"timed {args.steps} steps in {wall:.3f} s")
    stage.synchronize()

    # The kernel table and the roofline: the same K steps again with HIP events
    # around every op (per pass) and every library launch (per kernel class),
    # recorded on the stage's stream.
    profile = not args.no_profile
    events = [] if profile else None
    if profile:
        stage.profile_enable(True)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for i in range(args.steps):
            run_step(events)
        torch.cuda.synchronize()
        log(f"profiled {args.steps} steps in {time.perf_counter() - t1:.3f} s")
        stage.synchronize()

    F, B, W = cfg.flops_per_layer()
    it_flops = cfg.layers * cfg.n_mb * (F + B + W)
    ms_per_step = 1e3 * wall / args.steps
    out = {
        "metric": METRIC,
        "value": round(it_flops * args.steps / wall / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) activations, N(0,1e-2) upstream gradients)",
        "config": {"workload": workload_name(cfg), "layers": cfg.layers, "hidden": cfg.hidden,
                   "heads": cfg.heads, "ffn": cfg.ffn, "seq_len": cfg.seq,
                   "micro_batch": cfg.micro_batch, "micro_batches": cfg.n_mb,
                   "tokens_per_micro_batch": cfg.tokens, "parallelism": "one stage, one GPU",
                   "weight_pass_calls_per_step": sum(1 for k, _ in steps_ops if k == "W")},
        "mb_per_s": round(cfg.n_mb * args.steps / wall, 2),
        "pct_bf16_peak": round(100 * it_flops * args.steps / wall / 1e12 / PEAK_BF16_TFLOPS, 2),
    }
    if profile:
        per = {"F": 0.0, "B": 0.0, "W": 0.0, "STEP": 0.0}
        calls = {"F": [], "B": [], "W": []}  # TFLOP/s of each call (a W call may cover several micro-batches)
        pass_fl = {"F": F, "B": B, "W": W}
        for kind, a, b, nmb in events:
            ms = a.elapsed_time(b)
            per[kind] += ms
            if kind in calls and ms > 0:
                calls[kind].append(cfg.layers * nmb * pass_fl[kind] / (ms / 1e3) / 1e12)
        nl = cfg.layers * cfg.n_mb * args.steps
        out["pass_tflops"] = {k: round(nl * fl / (per[k] / 1e3) / 1e12, 2)
                              for k, fl in (("F", F), ("B", B), ("W", W))}
        out["pass_tflops_median"] = {k: round(float(np.median(v)), 2) for k, v in calls.items() if v}
        out["pass_ms_per_mb"] = {k: round(per[k] / (cfg.n_mb * args.steps), 3) for k in ("F", "B", "W")}
        out["optimizer_ms"] = round(per["STEP"] / args.steps, 3)
        prof = stage.profile_read()
        stage.profile_enable(False)
        kern = {}
        for name, r in prof.items():
            if r["launches"] == 0 or r["ms"] <= 0:
                continue
            e = {"launches": r["launches"], "avg_us": round(1e3 * r["ms"] / r["launches"], 2),
                 "share_pct": 0.0}
            if r["flops"] > 0:
                e["tflops"] = round(r["flops"] / (r["ms"] / 1e3) / 1e12, 2)
                e["pct_bf16_peak"] = round(100 * e["tflops"] / PEAK_BF16_TFLOPS, 2)
            if r["bytes"] > 0:
                e["gbs"] = round(r["bytes"] / (r["ms"] / 1e3) / 1e9, 1)
            kern[name] = e
        tot = sum(r["ms"] for r in prof.values())
        for name in kern:
            kern[name]["share_pct"] = round(100 * prof[name]["ms"] / tot, 1)
        out["kernels"] = kern
        dom = max(("gemm_fwd", "gemm_dgrad", "gemm_wgrad"), key=lambda n: prof[n]["ms"])
        r = prof[dom]
        achieved = r["flops"] / (r["ms"] / 1e3) / 1e12
        traffic, tsrc = measured_traffic(cfg, dom)
        out["roofline"] = {"kernel": f"{dom} (bf16 MFMA GEMM)", "bound": "mfma",
                           "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                           "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                           "traffic": traffic, "traffic_source": tsrc,
                           "avg_launch_us": round(1e3 * r["ms"] / r["launches"], 2),
                           "flops_per_launch": r["flops"] / r["launches"]}
    clocks = profile_clocks(cfg) if profile else {}
    if profile:
        for name, e in out["kernels"].items():
            ghz = clocks.get(name)
            if ghz and "tflops" in e:
                e["pct_bf16_peak_at_measured_clock"] = round(100 * e["tflops"] / (PEAK_PER_GHZ * ghz), 2)
        ghz = clocks.get(dom)
        rf = out["roofline"]
        rf["measured_clock_ghz"] = ghz
        rf["peak_at_measured_clock"] = round(PEAK_PER_GHZ * ghz, 1) if ghz else None
        rf["frac_at_measured_clock"] = round(rf["achieved"] / (PEAK_PER_GHZ * ghz), 4) if ghz else None
        rf["clock_source"] = clocks.get("_source")
    if not args.single_w and not args.no_single_w_leg and any(len(m) > 1 for k, m in steps_ops if k == "W"):
        # The same op list with one weight-pass call per micro-batch (the unit a
        # schedule defers into a single bubble): wall time of K steps, then the
        # same K steps with events for the weight pass and its GEMM class.
        plan = group(True)
        for _ in range(max(1, args.warmup)):
            run_step(plan=plan)
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        for _ in range(args.steps):
            run_step(plan=plan)
        torch.cuda.synchronize()
        wall1 = time.perf_counter() - t2
        leg = {"ms_per_step": round(1e3 * wall1 / args.steps, 3),
               "value": round(it_flops * args.steps / wall1 / 1e12, 2),
               "weight_pass_calls_per_step": sum(1 for k, _ in plan if k == "W")}
        if profile:
            ev = []
            stage.profile_enable(True)
            for _ in range(args.steps):
                run_step(ev, plan=plan)
            torch.cuda.synchronize()
            wms = sum(a.elapsed_time(b) for kind, a, b, _ in ev if kind == "W")
            leg["w_pass_tflops"] = round(cfg.layers * cfg.n_mb * args.steps * W / (wms / 1e3) / 1e12, 2)
            r = stage.profile_read()["gemm_wgrad"]
            stage.profile_enable(False)
            leg["gemm_wgrad"] = {"launches": r["launches"], "avg_us": round(1e3 * r["ms"] / r["launches"], 2),
                                 "tflops": round(r["flops"] / (r["ms"] / 1e3) / 1e12, 2)}
            leg["gemm_wgrad"]["pct_bf16_peak"] = round(100 * leg["gemm_wgrad"]["tflops"] / PEAK_BF16_TFLOPS, 2)
        out["single_w_leg"] = leg
        log(f"single weight-pass leg: {leg}")
    if not args.no_cpu_baseline:
        log("timing the fp64 CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(cfg, params)
    stage.close()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
