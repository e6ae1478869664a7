"""Summarise rocprofv3 output of a stage benchmark run into a short markdown
report with a machine-readable block that ``bench.py`` reads back.

Inputs (CSV files written by ``rocprofv3 --output-format csv``):
  --stats        ``*_kernel_stats.csv`` of ``rocprofv3 --kernel-trace --stats``
  --fetch/--write ``*_counter_collection.csv`` of ``rocprofv3 --pmc FETCH_SIZE``
                 and ``--pmc WRITE_SIZE`` runs of the same command
  --copy-fetch/--copy-write  the same counters over ``bench.py --copy-probe``
                 (plain 1 GiB device copies), which calibrate them: the
                 factor is (bytes the copy must move) / (bytes the counter
                 reports), applied to every kernel's reading.
  --mfma         ``*_counter_collection.csv`` of a ``rocprofv3 --pmc
                 SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16
                 GRBM_GUI_ACTIVE`` run of the same command: per kernel class
                 the matrix-core busy fraction (busy cycles over the 1024
                 SIMDs' active cycles), the bf16 MFMA flops executed (512 per
                 MOPS unit) and the sustained shader clock (GRBM_GUI_ACTIVE is
                 summed over the 8 XCDs, divided by the dispatch duration).
  --l2 / --l2-copy  ``*_counter_collection.csv`` of ``rocprofv3 --pmc
                 TCP_TCC_READ_REQ_sum TCP_TCC_READ_REQ_LATENCY_sum TCC_HIT_sum
                 TCC_MISS_sum GRBM_GUI_ACTIVE`` runs of the stage and of the
                 copy probe: per kernel class the L2 hit rate, the average
                 L1->L2 read latency, the read requests in flight per compute
                 unit (summed latency over active cycles) and the bytes per
                 clock each compute unit receives (request size calibrated on
                 the copy, whose reads are known).

Kernel names map to the stage library's kernel classes (the same classes its
per-launch profiler reports), so the per-launch averages here can be checked
against the benchmark's own event timing.

    python -m paper_2405_14009_amd.profile_summary --stats S.csv --fetch F.csv \\
        --write W.csv --copy-fetch CF.csv --copy-write CW.csv --bench bench.json \\
        --command "<commands>" --out profiles/<name>.md
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import sys
from collections import defaultdict

COPY_BYTES = 1 << 30  # per copy dispatch of bench.py --copy-probe (read and write)


_COMMENT = re.compile(r"//[^\n]*|/\*.*?\*/", re.S)


def code_text(src: str) -> str:
    """Source text without comments, trailing blanks and empty lines: what
    the compiler sees, so that editing a comment keeps the digest."""
    lines = (line.rstrip() for line in _COMMENT.sub("", src).splitlines())
    return "\n".join(line for line in lines if line)


def sources_digest(d: str = None) -> str:
    """sha256 over the code of the kernel and runtime sources (name + code
    text, sorted by name)."""
    d = d or os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
    h = hashlib.sha256()
    for name in sorted(os.listdir(d)):
        if name.endswith((".hip", ".h", ".cpp")):
            h.update(name.encode())
            with open(os.path.join(d, name), encoding="utf-8") as f:
                h.update(code_text(f.read()).encode())
    return h.hexdigest()


def kernel_class(name: str) -> str:
    # the one-tile and ping-pong bf16 GEMM kernels end their template arguments
    # with (A k-contiguous, B k-contiguous, epilogue); the persistent kernel
    # begins with (epilogue, A k-contiguous, B k-contiguous)
    m = re.search(r"gemm_bf16_persist_kernel<(\d+),\s*(true|false),\s*(true|false)(?:,\s*(?:true|false))?>", name)
    if m:
        epi, ak, bk = int(m.group(1)), m.group(2), m.group(3)
    else:
        m = re.search(r"gemm_bf16(?:_pp)?_kernel<[^>]*?(true|false),\s*(true|false),\s*(\d+)>", name)
        if m:
            ak, bk, epi = m.group(1), m.group(2), int(m.group(3))
    if m:
        if (ak, bk) == ("false", "false"):
            return "gemm_wgrad"
        if epi in (1, 2, 3):          # bias / bias + residual / bias + GeLU: the forward products
            return "gemm_fwd"
        if (ak, bk) == ("true", "true") and epi in (0, 4):
            return "gemm_dgrad"
        return "gemm_other"
    if "gemm_f32" in name:
        return "gemm_f32"
    if re.search(r"attn_fwd(_pair)?_k", name):
        return "attn_fwd"
    if "attn_bwd" in name:
        return "attn_bwd"
    if re.search(r"ln_(fwd|bwd)(_wave)?_k", name):
        return "layernorm"
    if "colsum" in name:
        return "reduce"
    if "adamw" in name:
        return "adamw"
    if "softmax" in name:
        return "softmax"
    if "copyBuffer" in name or "copy" in name.lower():
        return "copy"
    return "other"


def short(name: str) -> str:
    name = name.replace("(anonymous namespace)::", "").replace("void ", "")
    return name.split("(")[0] if "gemm" in name or "attn" in name else name[:90]


def read_stats(path):
    rows = []
    with open(path) as f:
        for r in csv.DictReader(f):
            rows.append({"name": r["Name"], "calls": int(r["Calls"]),
                         "total_ns": float(r["TotalDurationNs"]), "avg_ns": float(r["AverageNs"])})
    return rows


def read_counter(path, counter):
    """Per-dispatch values of one counter: list of (kernel name, value)."""
    out = []
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] == counter:
                out.append((r["Kernel_Name"], float(r["Counter_Value"])))
    return out


def calibrate(path, counter):
    vals = [v for n, v in read_counter(path, counter) if kernel_class(n) == "copy" or "elementwise" in n]
    vals = [v for v in vals if v > 0]
    if not vals:
        raise SystemExit(f"no copy dispatch with {counter} in {path}")
    big = max(vals)
    sel = [v for v in vals if v > 0.5 * big]  # the 1 GiB copies, not small helper launches
    kib = sum(sel) / len(sel)
    return COPY_BYTES / (kib * 1024.0), kib


CUS = 256
SIMDS = 1024     # 256 compute units x 4 SIMDs
XCDS = 8
FLOP_PER_CLK_SIMD = 1024   # dense bf16 MFMA


def mfma_classes(path):
    """Per kernel class: dispatches, summed duration, MFMA busy cycles, bf16
    MFMA flops and GUI-active cycles, from one counter pass."""
    disp = defaultdict(dict)
    with open(path) as f:
        for r in csv.DictReader(f):
            d = disp[r["Dispatch_Id"]]
            d["name"] = r["Kernel_Name"]
            d["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
            d[r["Counter_Name"]] = float(r["Counter_Value"])
    acc = defaultdict(lambda: {"n": 0, "ns": 0.0, "busy": 0.0, "mops": 0.0, "grbm": 0.0})
    for d in disp.values():
        if "GRBM_GUI_ACTIVE" not in d or d["ns"] <= 0:
            continue
        e = acc[kernel_class(d["name"])]
        e["n"] += 1
        e["ns"] += d["ns"]
        e["busy"] += d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        e["mops"] += d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)
        e["grbm"] += d["GRBM_GUI_ACTIVE"]
    out = {}
    for k, e in acc.items():
        cyc = e["grbm"] / XCDS                      # active cycles of one XCD
        out[k] = {"mfma_busy_pct": round(100 * e["busy"] / (cyc * SIMDS), 2) if cyc else None,
                  "mfma_bf16_flops_per_dispatch": round(512 * e["mops"] / e["n"]),
                  "mfma_bf16_tflops_executed": round(512 * e["mops"] / e["ns"] / 1e3, 1)}
        # the counter window exceeds a dispatch by microseconds, so the clock is
        # read only off the matrix-core classes' dispatches of 40 us or more
        # (the classes whose peak it scales)
        if e["mops"] > 0 and e["ns"] / e["n"] >= 40e3:
            out[k]["sclk_ghz"] = round(cyc / e["ns"], 3)
    return out


def l2_classes(path, copy_path=None):
    """Per kernel class from one L2 counter pass (see --l2)."""
    disp = defaultdict(dict)
    with open(path) as f:
        for r in csv.DictReader(f):
            d = disp[r["Dispatch_Id"]]
            d["name"] = r["Kernel_Name"]
            d[r["Counter_Name"]] = float(r["Counter_Value"])
    req_bytes = None
    if copy_path:
        reqs = [v for n, v in read_counter(copy_path, "TCP_TCC_READ_REQ_sum")
                if kernel_class(n) == "copy" or "elementwise" in n]
        if reqs:
            big = max(reqs)
            sel = [v for v in reqs if v > 0.5 * big]
            req_bytes = COPY_BYTES / (sum(sel) / len(sel))
    acc = defaultdict(lambda: defaultdict(float))
    for d in disp.values():
        if "GRBM_GUI_ACTIVE" not in d:
            continue
        e = acc[kernel_class(d["name"])]
        for c in ("TCP_TCC_READ_REQ_sum", "TCP_TCC_READ_REQ_LATENCY_sum", "TCC_HIT_sum", "TCC_MISS_sum",
                  "GRBM_GUI_ACTIVE"):
            e[c] += d.get(c, 0.0)
    out = {}
    for k, e in acc.items():
        req, lat = e["TCP_TCC_READ_REQ_sum"], e["TCP_TCC_READ_REQ_LATENCY_sum"]
        cyc = e["GRBM_GUI_ACTIVE"] / XCDS
        hm = e["TCC_HIT_sum"] + e["TCC_MISS_sum"]
        if not req or not cyc:
            continue
        o = {"l2_hit_pct": round(100 * e["TCC_HIT_sum"] / hm, 1) if hm else None,
             "l1_l2_read_latency_cycles": round(lat / req, 1),
             "read_requests_in_flight_per_cu": round(lat / (cyc * CUS), 1),
             "read_requests_per_clk_per_cu": round(req / (cyc * CUS), 3)}
        if req_bytes:
            o["read_request_bytes"] = round(req_bytes, 1)
            o["read_bytes_per_clk_per_cu"] = round(req * req_bytes / (cyc * CUS), 2)
        out[k] = o
    return out


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--stats", required=True)
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-fetch")
    ap.add_argument("--copy-write")
    ap.add_argument("--mfma")
    ap.add_argument("--l2")
    ap.add_argument("--l2-copy")
    ap.add_argument("--bench", help="bench.py JSON line of the same build")
    ap.add_argument("--command", required=True, help="the commands that produced the inputs")
    ap.add_argument("--title", default="GPT-6.7B-shaped stage iteration")
    ap.add_argument("--out", required=True)
    a = ap.parse_args(argv)

    stats = read_stats(a.stats)
    tot = sum(r["total_ns"] for r in stats)
    cls = defaultdict(lambda: {"calls": 0, "total_ns": 0.0})
    for r in stats:
        c = cls[kernel_class(r["name"])]
        c["calls"] += r["calls"]
        c["total_ns"] += r["total_ns"]

    traffic = {}
    cal = {}
    if a.fetch and a.write and a.copy_fetch and a.copy_write:
        ff, fk = calibrate(a.copy_fetch, "FETCH_SIZE")
        fw, wk = calibrate(a.copy_write, "WRITE_SIZE")
        cal = {"fetch_factor": round(ff, 4), "write_factor": round(fw, 4),
               "copy_fetch_kib": round(fk, 1), "copy_write_kib": round(wk, 1),
               "copy_bytes": COPY_BYTES}
        acc = defaultdict(lambda: [0.0, 0.0, 0, 0])
        for n, v in read_counter(a.fetch, "FETCH_SIZE"):
            e = acc[kernel_class(n)]
            e[0] += v * 1024.0 * ff
            e[2] += 1
        for n, v in read_counter(a.write, "WRITE_SIZE"):
            e = acc[kernel_class(n)]
            e[1] += v * 1024.0 * fw
            e[3] += 1
        for k, (fb, wb, nf, nw) in acc.items():
            if nf and nw:
                traffic[k] = {"fetch_bytes_per_dispatch": fb / nf, "write_bytes_per_dispatch": wb / nw,
                              "bytes_per_dispatch": fb / nf + wb / nw}

    mfma = mfma_classes(a.mfma) if a.mfma else {}
    l2 = l2_classes(a.l2, a.l2_copy) if a.l2 else {}

    bench = None
    if a.bench:
        with open(a.bench) as f:
            for line in f:
                line = line.strip()
                if line.startswith("{"):
                    bench = json.loads(line)

    L = [f"# Kernel time and HBM traffic: {a.title}", ""]
    L += ["Commands (from the repository root on one MI355X; `$R` is the repository path):", "", "```",
          a.command.strip(), "```", ""]
    L += ["| kernel class | dispatches | avg us / dispatch | % time | HBM bytes / dispatch (calibrated) |",
          "|---|---:|---:|---:|---:|"]
    for k, c in sorted(cls.items(), key=lambda kv: -kv[1]["total_ns"]):
        t = traffic.get(k)
        tb = f"{t['bytes_per_dispatch'] / 1e6:.1f} MB" if t else "—"
        L.append(f"| {k} | {c['calls']} | {c['total_ns'] / c['calls'] / 1e3:.1f} | "
                 f"{100 * c['total_ns'] / tot:.1f} | {tb} |")
    L += ["", "Top kernels:", "", "| kernel | calls | avg us | % time |", "|---|---:|---:|---:|"]
    for r in sorted(stats, key=lambda r: -r["total_ns"])[:14]:
        L.append(f"| `{short(r['name'])}` | {r['calls']} | {r['avg_ns'] / 1e3:.1f} | "
                 f"{100 * r['total_ns'] / tot:.2f} |")
    if mfma:
        L += ["", "Matrix cores (one counter pass: SQ_VALU_MFMA_BUSY_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_BF16, "
              "GRBM_GUI_ACTIVE).  Busy % is MFMA busy cycles over the 1024 SIMDs' active cycles; the "
              "clock is the XCDs' active cycles over the dispatch duration; the peak at that clock is "
              "1024 SIMDs x 1024 flop/clk x clock:", "",
              "| kernel class | MFMA busy % | bf16 MFMA TFLOP executed / dispatch | executed TFLOP/s | "
              "sustained clock (GHz) | dense bf16 peak at that clock (TFLOP/s) |",
              "|---|---:|---:|---:|---:|---:|"]
        for k, e in sorted(mfma.items(), key=lambda kv: -cls[kv[0]]["total_ns"] if kv[0] in cls else 0):
            if not e["mfma_bf16_flops_per_dispatch"] or "sclk_ghz" not in e:
                continue
            L.append(f"| {k} | {e['mfma_busy_pct']} | {e['mfma_bf16_flops_per_dispatch'] / 1e12:.4f} | "
                     f"{e['mfma_bf16_tflops_executed']} | {e['sclk_ghz']} | "
                     f"{SIMDS * FLOP_PER_CLK_SIMD * e['sclk_ghz'] / 1e3:.0f} |")
    if l2:
        L += ["", "L1 -> L2 reads (one counter pass: TCP_TCC_READ_REQ_sum, TCP_TCC_READ_REQ_LATENCY_sum, "
              "TCC_HIT_sum, TCC_MISS_sum, GRBM_GUI_ACTIVE).  In flight = summed request latency over the "
              "256 compute units' active cycles; bytes per clock use the request size measured on the copy "
              "probe:", "",
              "| kernel class | L2 hit % | average L1->L2 read latency (cycles) | read requests in flight per CU "
              "| read bytes / clk / CU |", "|---|---:|---:|---:|---:|"]
        for k, e in sorted(l2.items(), key=lambda kv: -cls[kv[0]]["total_ns"] if kv[0] in cls else 0):
            if k not in cls or cls[k]["total_ns"] < 0.005 * tot:
                continue
            L.append(f"| {k} | {e['l2_hit_pct']} | {e['l1_l2_read_latency_cycles']} | "
                     f"{e['read_requests_in_flight_per_cu']} | {e.get('read_bytes_per_clk_per_cu', '—')} |")
    if cal:
        L += ["", f"Counter calibration (plain 1 GiB device copies): FETCH_SIZE reads "
              f"{cal['copy_fetch_kib']:.0f} KiB and WRITE_SIZE {cal['copy_write_kib']:.0f} KiB per copy "
              f"of {COPY_BYTES // 1024} KiB; factors {cal['fetch_factor']} (fetch) and "
              f"{cal['write_factor']} (write) scale every reading above."]
    if bench:
        k = bench.get("kernels", {})
        L += ["", f"bench.py line of the same build: value {bench['value']} {bench['unit']}, "
              f"{bench.get('mb_per_s')} micro-batches/s; event-timed average per launch: " +
              ", ".join(f"{n} {v['avg_us']} us" for n, v in k.items() if n.startswith("gemm"))]
    block = {"sources_sha256": sources_digest(), "classes": {}, "calibration": cal}
    for k, c in cls.items():
        e = {"dispatches": c["calls"], "avg_us": round(c["total_ns"] / c["calls"] / 1e3, 2)}
        if k in traffic:
            e.update({kk: round(v) for kk, v in traffic[k].items()})
        if k in mfma:
            e.update(mfma[k])
        if k in l2:
            e.update(l2[k])
        block["classes"][k] = e
    L += ["", "Machine-readable (read by bench.py; `sources_sha256` is the digest of the kernel "
          "sources these counters were taken with):", "", "```json", json.dumps(block, indent=1), "```", ""]
    with open(a.out, "w") as f:
        f.write("\n".join(L))
    print(f"wrote {a.out}")
    return 0


if __name__ == "__main__":
    sys.exit(main())
