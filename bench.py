#!/usr/bin/env python3
"""Tree-verification step benchmark on one MI355X.

A step is one pass of the whole hot path over one batch: tree-masked GQA
attention of all draft-tree nodes (one attention layer at the workload's
shape) followed by greedy tree acceptance over the nodes' target logits.
Inputs are seeded synthetic tensors of the workload's shape, resident in HBM
before timing starts.  Each timed graph rotates over enough input replicas
that at least 512 MB (twice the MI355X last-level cache) is touched between
two uses of one replica, so every timed call reads its inputs from HBM; the
JSON labels each group of timings with its reuse distance.

The headline workload is the largest configuration (big_tree_32b: Qwen3-32B
attention geometry, one sequence, 8192 cached rows, a 512-node tree).  Every
one of the five workloads is also measured the same way and reported in
``detail.per_config``: step, attention and acceptance times, tree-tokens/s,
the roofline position of each kernel, and the error of the timed outputs
against the CPU oracle on a sample.

Prints one JSON line: tree-tokens/s (B*N / step time) of the headline, ms
per step, the roofline position of the dominant kernel (algorithmic bytes or
flops over its event-timed duration) and the CPU oracle's throughput on a
bounded sample.
"""
from __future__ import annotations

import os

# The CPU leg's thread count is pinned before numpy loads its BLAS: the
# environment's value if set, else every CPU this process may run on.
AFFINITY_CPUS = len(os.sched_getaffinity(0))
THREAD_VARS = ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")
for _v in THREAD_VARS:
    os.environ.setdefault(_v, str(AFFINITY_CPUS))

import argparse  # noqa: E402
import hashlib  # noqa: E402
import json  # noqa: E402
import sys  # noqa: E402
import time  # noqa: E402

import numpy as np  # noqa: E402

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
MALL_BYTES = 256 << 20
MAX_REPLICAS = 4096            # bounds graph size and capture time at the smallest shapes
PAGE_BLOCK = 64                # rows per paged-cache block in the paged timing
TRAIN_ANCHORS, TRAIN_BLOCK, TRAIN_CONTEXT = 512, 16, 4096   # training-mask attention timing
HEADLINE = "big_tree_32b"
WORKLOAD_ORDER = ["tiny", "qwen3_8b", "long_ctx", "batched_30b_a3b", "big_tree_32b"]
CHECK_NODES = 16               # nodes per sequence whose timed output the oracle checks


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--settle-ms", type=float, default=200.0,
                    help="untimed replays of each timed graph for at least this long before its "
                         "timed region, so the GPU clock has left its idle ramp")
    ap.add_argument("--workload", default=HEADLINE,
                    help="headline workload (default: the largest, big_tree_32b)")
    ap.add_argument("--core-only", action="store_true",
                    help="time only the headline workload's step, attention and acceptance "
                         "(no other workloads, no extra paths, no CPU leg): the profiler runs")
    ap.add_argument("--replicas", type=int, default=0, help="0 = enough that every timed graph touches 2x the LLC between reuses")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the CPU leg (oracle timing and the oracle checks)")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    ap.add_argument("--copy-only", action="store_true",
                    help="only run 10 plain device copies of 256 MiB (calibrates the HBM "
                         "traffic counters: each copy reads and writes exactly 256 MiB)")
    ap.add_argument("--kernel", default="attn_main", choices=["attn_main", "accept_scan"],
                    help="kernel family the --summarize-traffic summary covers")
    ap.add_argument("--summarize-traffic", nargs=4, default=None,
                    metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                    help="no GPU: turn the counter CSVs of four rocprofv3 --pmc runs (FETCH_SIZE "
                         "and WRITE_SIZE of this benchmark, then of --copy-only) into "
                         "profiles/traffic_<kernel>_<workload>.json and .md")
    ap.add_argument("--summarize-counters", nargs="+", default=None, metavar="PMC_DIR",
                    help="no GPU: turn rocprofv3 --pmc runs of this benchmark (one or more "
                         "output directories) into profiles/counters_attn_main_<workload>.md")
    ap.add_argument("--summarize-trace", nargs=2, default=None, metavar=("TRACE_DIR", "BENCH_LOG"),
                    help="no GPU: turn a rocprofv3 --kernel-trace --stats run of this benchmark and "
                         "the log of the same command run without the profiler into "
                         "profiles/kernel_trace_<workload>.md")
    return ap.parse_args()


COPY_BYTES = 256 << 20


def _counter_rows(d, counter):
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            rows += [r for r in csv.DictReader(fh) if r["Counter_Name"] == counter]
    if not rows:
        raise SystemExit(f"no {counter} rows under {d}")
    return rows


KERNEL_PATTERNS = {
    # the verification launch is the contiguous-cache instantiation with the
    # most dispatches (the other timed paths launch fewer)
    # (template arguments D, WR, WK, NS, paged, shared queries)
    "attn_main": (r"attn_main<(\d+), (\d+), (\d+), (\d+), false(?:, (?:false|true))?>",
                  "attn_main<%s,%s,%s,%s>"),
    "accept_scan": (r"accept_scan<(\w+), (\w+)>", "accept_scan<%s,%s>"),
}


def summarize_traffic(dirs, workload, kernel_family):
    """HBM bytes per launch of one kernel from FETCH_SIZE / WRITE_SIZE (KiB
    per dispatch), each scaled by what the same counter reads for a 256 MiB
    device copy."""
    import re
    import statistics
    pat = re.compile(KERNEL_PATTERNS[kernel_family][0])
    fmt = KERNEL_PATTERNS[kernel_family][1]
    med, names, n = {}, set(), {}
    for d, c in zip(dirs[:2], ["FETCH_SIZE", "WRITE_SIZE"]):
        by = {}
        for r in _counter_rows(d, c):
            m = pat.search(r["Kernel_Name"])
            if m:
                by.setdefault(fmt % m.groups(), []).append(float(r["Counter_Value"]))
        if not by:
            raise SystemExit(f"no {kernel_family} dispatches in {d}")
        name = max(by, key=lambda k: len(by[k]))
        names.add(name)
        med[c], n[c] = statistics.median(by[name]), len(by[name])
    if len(names) != 1:
        raise SystemExit(f"the two counter runs disagree on the kernel: {sorted(names)}")
    cal = {}
    for d, c in zip(dirs[2:], ["FETCH_SIZE", "WRITE_SIZE"]):
        vals = [float(r["Counter_Value"]) for r in _counter_rows(d, c)
                if "copyBuffer" in r["Kernel_Name"] or "copy" in r["Kernel_Name"].lower()]
        cal[c] = statistics.median(vals)
    kib = COPY_BYTES / 1024
    fs, ws = kib / cal["FETCH_SIZE"], kib / cal["WRITE_SIZE"]
    fetch_b = med["FETCH_SIZE"] * fs * 1024
    write_b = med["WRITE_SIZE"] * ws * 1024
    kernel = names.pop()
    rec = {"kernel": kernel, "workload": workload,
           "fetch_kib_per_dispatch": med["FETCH_SIZE"], "write_kib_per_dispatch": med["WRITE_SIZE"],
           "dispatches": n,
           "copy_calibration": {"bytes": COPY_BYTES, "fetch_kib": cal["FETCH_SIZE"],
                                "write_kib": cal["WRITE_SIZE"], "fetch_scale": round(fs, 4),
                                "write_scale": round(ws, 4)},
           "hbm_bytes_per_launch": int(round(fetch_b + write_b)),
           "kernel_src_sha": kernel_source_sha()}
    base = os.path.join(ROOT, "profiles", f"traffic_{kernel_family}_{workload}")
    with open(base + ".json", "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    with open(base + ".md", "w") as fh:
        fh.write(f"""# HBM traffic: {kernel}, workload {workload}

Commands (repository root, rocprofv3 run from /tmp with TMPDIR=/tmp; one counter per run):

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d <f> -o b -- python3 bench.py --workload {workload} --core-only --steps 20 --warmup 3
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d <w> -o b -- python3 bench.py --workload {workload} --core-only --steps 20 --warmup 3
    rocprofv3 --pmc FETCH_SIZE --output-format csv -d <cf> -o c -- python3 bench.py --copy-only
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d <cw> -o c -- python3 bench.py --copy-only
    python3 bench.py --workload {workload} --kernel {kernel_family} --summarize-traffic <f> <w> <cf> <cw>

Calibration: a plain {COPY_BYTES >> 20} MiB device copy reads FETCH_SIZE = {cal['FETCH_SIZE']:.1f} KiB
and WRITE_SIZE = {cal['WRITE_SIZE']:.1f} KiB per dispatch against {kib:.0f} KiB moved each way, so
the scale factors are {fs:.4f} (fetch) and {ws:.4f} (write).

| counter | raw KiB / dispatch (median of {n['FETCH_SIZE']}) | scaled MB |
|---|---|---|
| FETCH_SIZE | {med['FETCH_SIZE']:.1f} | {fetch_b / 1e6:.2f} |
| WRITE_SIZE | {med['WRITE_SIZE']:.1f} | {write_b / 1e6:.2f} |
| total | | {(fetch_b + write_b) / 1e6:.2f} |
""")
    print(json.dumps(rec))


SIMDS = 256 * 4        # MI355X: 256 CUs of 4 SIMDs
CLOCK_HZ = 2.4e9


def summarize_counters(dirs, workload):
    """Per-dispatch medians of SQ counters of the verification attention
    kernel (the contiguous-cache instantiation with the most dispatches) and
    the utilisations they imply."""
    import csv
    import glob
    import re
    import statistics
    pat = re.compile(KERNEL_PATTERNS["attn_main"][0])
    vals, durs = {}, {}
    for d in dirs:
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(f) as fh:
                for r in csv.DictReader(fh):
                    m = pat.search(r["Kernel_Name"])
                    if not m:
                        continue
                    k = "attn_main<%s,%s,%s,%s>" % m.groups()
                    vals.setdefault(k, {}).setdefault(r["Counter_Name"], []).append(
                        float(r["Counter_Value"]))
                    durs.setdefault(k, []).append(
                        (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    if not vals:
        raise SystemExit("no attn_main dispatches in the counter runs")
    kernel = max(vals, key=lambda k: len(durs[k]))
    c = {n: statistics.median(v) for n, v in vals[kernel].items()}
    t = statistics.median(durs[kernel])
    lines = [f"# SQ counters: {kernel}, workload {workload}", "",
             "Commands (repository root, rocprofv3 run from /tmp with TMPDIR=/tmp; each --pmc "
             "set in a run of its own):", ""]
    sets = ["SQ_WAVES SQ_BUSY_CYCLES SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU SQ_INSTS_MFMA "
            "SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT SQ_ACTIVE_INST_LDS",
            "SQ_WAIT_INST_ANY SQ_ACTIVE_INST_VALU SQ_WAIT_ANY SQ_ACTIVE_INST_ANY "
            "SQ_WAIT_INST_LDS SQ_LDS_IDX_ACTIVE"]
    for cs in sets:
        lines.append(f"    rocprofv3 --pmc {cs} --output-format csv -d <out> -o p -- python3 "
                     f"bench.py --workload {workload} --core-only --steps 20 --warmup 2")
    lines += [f"    python3 bench.py --workload {workload} --summarize-counters <out> <out2>", "",
              f"Median over {len(durs[kernel])} counter-run dispatches of the kernel; its median "
              f"duration in those runs is {t * 1e6:.1f} us.", "",
              "| counter | median per dispatch |", "|---|---|"]
    for n in sorted(c):
        lines.append(f"| {n} | {c[n]:.0f} |")
    lines += ["", "Derived (MI355X: 1024 SIMDs, 2.4 GHz; SQ_BUSY_CYCLES summed over the 32 "
              "shader engines of 32 SIMDs):", ""]
    if "SQ_VALU_MFMA_BUSY_CYCLES" in c:
        mb = c["SQ_VALU_MFMA_BUSY_CYCLES"]
        lines.append(f"* matrix cores busy: {100 * mb / (SIMDS * CLOCK_HZ * t):.1f}% of the "
                     f"kernel's SIMD-cycles")
        if "SQ_BUSY_CYCLES" in c:
            lines.append(f"* matrix cores busy: {100 * mb / (c['SQ_BUSY_CYCLES'] * 32):.1f}% of "
                         f"the cycles the shader engines were busy")
    if "SQ_INSTS_MFMA" in c and "SQ_INSTS_VALU" in c:
        lines.append(f"* VALU instructions (MFMA included) per MFMA: "
                     f"{c['SQ_INSTS_VALU'] / c['SQ_INSTS_MFMA']:.2f}")
    if "SQ_LDS_BANK_CONFLICT" in c and "SQ_LDS_IDX_ACTIVE" in c:
        lines.append(f"* LDS bank-conflict cycles per LDS-active cycle: "
                     f"{c['SQ_LDS_BANK_CONFLICT'] / c['SQ_LDS_IDX_ACTIVE']:.2f}")
    if "SQ_LDS_IDX_ACTIVE" in c:
        lines.append(f"* LDS active: {100 * c['SQ_LDS_IDX_ACTIVE'] / (256 * CLOCK_HZ * t):.1f}% "
                     f"of the kernel's CU-cycles")
    if "SQ_WAIT_INST_ANY" in c and "SQ_ACTIVE_INST_ANY" in c:
        lines.append(f"* wave cycles waiting for a dependency per issuing cycle: "
                     f"{c['SQ_WAIT_INST_ANY'] / c['SQ_ACTIVE_INST_ANY']:.2f}")
    path = os.path.join(ROOT, "profiles", f"counters_attn_main_{workload}.md")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    # the matrix-core busy fraction for the bench line, with the sources'
    # hash so that it is reported only while it describes the running code
    if "SQ_VALU_MFMA_BUSY_CYCLES" in c:
        rec = {"kernel": kernel, "workload": workload, "dispatches": len(durs[kernel]),
               "median_us": round(t * 1e6, 2),
               "mfma_busy_frac": round(c["SQ_VALU_MFMA_BUSY_CYCLES"] / (SIMDS * CLOCK_HZ * t), 4),
               "kernel_src_sha": kernel_source_sha()}
        with open(path[:-3] + ".json", "w") as fh:
            json.dump(rec, fh, indent=1)
            fh.write("\n")
    print(path)


def summarize_trace(trace_dir, bench_log, workload):
    """Kernel-time table from rocprofv3's kernel stats, beside the event-timed
    figures of the same command run without the profiler."""
    import csv
    import glob
    files = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)
    if len(files) != 1:
        raise SystemExit(f"expected one kernel_stats.csv under {trace_dir}, got {files}")
    with open(files[0]) as fh:
        rows = list(csv.DictReader(fh))
    durs = {}
    for f in glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                durs.setdefault(r["Kernel_Name"], []).append(
                    (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3)
    line = None
    with open(bench_log) as fh:
        for ln in fh:
            if ln.startswith("{") and '"metric"' in ln:
                line = json.loads(ln)
    if line is None or line["config"]["workload"] != workload:
        raise SystemExit(f"no bench line for {workload} in {bench_log}")
    c, d = line["config"], line["detail"]
    pc = d["per_config"][workload]
    out = [f"# Kernel trace: workload {workload} (B={c['B']}, Hq={c['Hq']}, Hkv={c['Hkv']}, "
           f"D={c['D']}, L={c['Lmax']}, N={c['N']}, V={c['V']} {c['logits']})", "",
           "Command (repository root; rocprofv3 run from /tmp with TMPDIR=/tmp):", "",
           f"    rocprofv3 --kernel-trace --stats --output-format csv -d <out> -o bench -- "
           f"python3 bench.py --workload {workload} --core-only",
           f"    python3 bench.py --workload {workload} --summarize-trace <out> <log of the same "
           f"bench.py command without the profiler>", "",
           "Calls include warm-up, graph capture and every timed graph (step, attention alone, "
           "acceptance alone).", "",
           "| kernel | calls | avg us | median us | p10 us | p90 us | min us | max us | "
           "% of GPU time |",
           "|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        name = r["Name"] if len(r["Name"]) <= 72 else r["Name"][:69] + "..."
        dv = np.array(durs.get(r["Name"], [float("nan")]))
        out.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                   f"{np.median(dv):.2f} | {np.percentile(dv, 10):.2f} | "
                   f"{np.percentile(dv, 90):.2f} | "
                   f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                   f"{float(r['Percentage']):.2f} |")
    out += ["", "Same command without the profiler (HIP events around graph replays on the "
            "launch stream):", "",
            f"    step {pc['us_per_step']:.2f} us = attention {pc['attention_us']:.2f} us + "
            f"acceptance {pc['accept_us']:.2f} us", ""]
    path = os.path.join(ROOT, "profiles", f"kernel_trace_{workload}.md")
    with open(path, "w") as fh:
        fh.write("\n".join(out))
    print(path)


def copy_only():
    import torch
    dev = torch.device("cuda:0")
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "copies": 10}), flush=True)


def depths(parent_row):
    d = np.zeros(len(parent_row), dtype=np.int64)
    for i in range(1, len(parent_row)):
        d[i] = d[parent_row[i]] + 1
    return d


def algorithmic_work(inp, w):
    """Bytes and flops the method must move/compute (no padding, no dense
    tree tile): KV rows < kv_len once, q/out/tree K/V once; 4*D flops per
    (query head, visible key) pair."""
    B, N, Hq, Hkv, D = w.B, w.N, w.Hq, w.Hkv, w.D
    kv = inp["kv_len"].astype(np.int64)
    vis = sum(int(kv[b]) * N + int((depths(inp["parent"][b]) + 1).sum()) for b in range(B))
    attn_bytes = int(kv.sum()) * Hkv * D * 2 * 2 + 2 * B * N * Hq * D * 2 + \
        2 * B * N * Hkv * D * 2 + B * N * 4 + B * 4
    attn_flops = 4 * D * Hq * vis
    esize = 4 if w.logits_dtype == "f32" else 2
    acc_bytes = B * N * w.V * esize + 2 * B * N * 4 + B * (w.Dmax + N + 1) * 4
    return attn_bytes, attn_flops, acc_bytes


def kernel_source_sha():
    h = hashlib.sha256()
    for f in ["tv_attention.hip", "tv_accept.hip", "tv_plan.h", "tv_walk.h", "tv_stream.h"]:
        with open(os.path.join(ROOT, "paper_2606_18394_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload):
    """HBM bytes per launch from committed rocprofv3 counter summaries, only
    if they were taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("kernel_src_sha") != kernel_source_sha():
        return None
    return rec.get("hbm_bytes_per_launch")


def measured_mfma_busy(workload):
    """Fraction of the attention kernel's SIMD-cycles its matrix cores were
    busy (SQ_VALU_MFMA_BUSY_CYCLES from committed rocprofv3 counter runs), only
    if they were taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"counters_attn_main_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("kernel_src_sha") != kernel_source_sha():
        return None
    return rec.get("mfma_busy_frac")


def roofline(name, t_s, nbytes, flops, kernel, workload):
    """Position of one kernel against the roofline that binds it: HBM bytes
    or bf16 MFMA flops at the MI355X peaks, whichever takes longer."""
    if flops == 0 or nbytes / (HBM_PEAK_GBS * 1e9) >= flops / (BF16_PEAK_TFLOPS * 1e12):
        r = {"bound": "hbm", "achieved": nbytes / t_s / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    else:
        r = {"bound": "mfma", "achieved": flops / t_s / 1e12, "peak": BF16_PEAK_TFLOPS,
             "unit": "TFLOP/s"}
    r["frac"] = r["achieved"] / r["peak"]
    r["kernel"] = name
    r["traffic"] = measured_traffic(kernel, workload)
    if kernel == "attn_main" and r["bound"] == "mfma":
        r["mfma_busy"] = measured_mfma_busy(workload)
    return r


# --------------------------------------------------------------------- CPU leg

def _thread_report():
    try:
        from threadpoolctl import threadpool_info
        blas = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:
        blas = None
    return blas, {v: os.environ.get(v) for v in THREAD_VARS}


def cpu_baseline(inp, w, draft, budget_s):
    """The oracle, as it stands, timed on a bounded sample of the same step
    (and its attention sample compared with nothing: timing only)."""
    import oracle
    blas, env = _thread_report()
    q = oracle.decode_bf16(inp["q"])
    kc, vc = oracle.decode_bf16(inp["k_cache"]), oracle.decode_bf16(inp["v_cache"])
    kt, vt = oracle.decode_bf16(inp["k_tree"]), oracle.decode_bf16(inp["v_tree"])
    # attention on a growing node sample until the budget's first half is used
    n_nodes, t_attn = 0, 0.0
    rng = np.random.default_rng(0)
    order = rng.permutation(w.N)
    while n_nodes < w.N and t_attn < budget_s / 2:
        k = min(max(1, w.N // 16), w.N - n_nodes)
        nodes = np.sort(order[n_nodes:n_nodes + k])
        t0 = time.perf_counter()
        oracle.tree_attention(q, kc, vc, kt, vt, inp["parent"], inp["kv_len"], nodes=nodes)
        t_attn += time.perf_counter() - t0
        n_nodes += k
    attn_step = t_attn * w.N / n_nodes
    lg = inp["logits"] if w.logits_dtype == "f32" else oracle.decode_bf16(inp["logits"])
    t0 = time.perf_counter()
    oracle.tree_accept(lg, draft, inp["parent"], w.Dmax)
    acc_step = time.perf_counter() - t0
    step = attn_step + acc_step
    return {"value": w.B * w.N / step, "unit": "tree-tokens/s",
            "cores": int(blas) if blas else AFFINITY_CPUS, "kind": "oracle",
            "affinity_cpus": AFFINITY_CPUS, "blas_threads": blas, "thread_env": env,
            "us_per_step": step * 1e6,
            "sample": f"attention on {n_nodes}/{w.N} nodes x all {w.Hq} heads of batch {w.B} "
                      f"({t_attn:.1f} s, scaled to all nodes) + full acceptance "
                      f"({acc_step:.1f} s); fp64 numpy, BLAS on {blas} threads, elementwise "
                      f"work on one"}


def oracle_check(inp, w, draft, got_rows, nodes, acc):
    """The timed outputs against the oracle: attention on the sampled nodes
    (all heads) as max-abs error, acceptance bit for bit."""
    import oracle
    dec = oracle.decode_bf16
    err = 0.0
    for b in range(w.B):
        ref = oracle.tree_attention(dec(inp["q"][b:b + 1]), dec(inp["k_cache"][b:b + 1]),
                                    dec(inp["v_cache"][b:b + 1]), dec(inp["k_tree"][b:b + 1]),
                                    dec(inp["v_tree"][b:b + 1]), inp["parent"][b:b + 1],
                                    inp["kv_len"][b:b + 1], nodes=nodes[b])[0]
        err = max(err, float(np.abs(got_rows[b] - ref).max()))
    lg = inp["logits"] if w.logits_dtype == "f32" else dec(inp["logits"])
    rl, rp, rt = oracle.tree_accept(lg, draft, inp["parent"], w.Dmax)
    exact = bool(np.array_equal(acc[0], rl) and np.array_equal(acc[1], rp) and
                 np.array_equal(acc[2], rt))
    return {"attention_max_abs_err": err,
            "attention_rows_checked": int(sum(len(n) for n in nodes) * w.Hq),
            "accept_bit_exact": exact}


def check_nodes(parent_row, k, seed):
    """Nodes whose timed attention output the oracle checks: the root, the
    last node, the deepest node and a seeded sample."""
    N = len(parent_row)
    d = depths(parent_row)
    pick = {0, N - 1, int(np.argmax(d))}
    pick |= set(np.random.default_rng(seed).choice(N, size=min(k, N), replace=False).tolist())
    return np.array(sorted(pick))


# --------------------------------------------------------------------- GPU

def _bf(torch, dev, a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)


def _i32(torch, dev, a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)


class Timer:
    """HIP graphs of a path's launches, replayed between HIP events on the
    stream the graphs are launched on.  A graph's R calls take R different
    input replicas in turn; k timed calls are k // R replays of that graph
    and one replay of a graph of its first k % R calls, so exactly k calls
    are timed and the timed region measures the GPU, not Python's launch
    overhead.  Untimed replays come first, for at least `settle_s` seconds:
    the shader clock ramps up over the first tens of milliseconds of work
    after the GPU has idled (graph capture idles it), and the timed region
    should see the clock a continuously running step sees.  They end with a
    whole replay, so the first timed call finds its replica least recently
    used."""

    def __init__(self, torch, R, settle_s=0.2):
        self.torch, self.R, self.graphs, self.settle_s = torch, R, {}, settle_s

    def _cap(self, fn, rs):
        g = self.torch.cuda.CUDAGraph()
        with self.torch.cuda.graph(g):
            for r in rs:
                fn(r)
        return g

    def capture(self, name, fn, R=None):
        R = R or self.R
        self.graphs[name] = (fn, R, self._cap(fn, range(R)), {})

    def time_ms(self, name, k):
        torch = self.torch
        fn, R, full, heads = self.graphs[name]
        rem = k % R
        if rem and rem not in heads:
            heads[rem] = self._cap(fn, range(rem))
        t0 = time.perf_counter()
        n = 0
        while n < 2 or time.perf_counter() - t0 < self.settle_s:   # untimed replays
            full.replay()
            n += 1
            if n % 8 == 0:
                torch.cuda.synchronize()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(k // R):
            full.replay()
        if rem:
            heads[rem].replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / k     # ms


def replicas_for(nbytes):
    """Input replicas one timed graph rotates over so that at least twice
    the last-level cache is touched between two uses of one replica: every
    timed call then reads its inputs from HBM."""
    return max(1, min(MAX_REPLICAS, -(-2 * MALL_BYTES // max(1, nbytes))))


def cache_state(reuse):
    """Label of the timed graphs' cache state from the bytes each touches
    between two uses of one input replica."""
    warm = [nm for nm, b in reuse.items() if b < 2 * MALL_BYTES]
    mb = ", ".join(f"{nm} {b / 2**20:.0f} MiB" for nm, b in reuse.items())
    if not warm:
        return f"cold: every replica reused after >= 2x the 256 MiB LLC ({mb})"
    return f"warm in the 256 MiB LLC: {', '.join(warm)} (reuse distance {mb})"


def run_workload(name, args, extras, cpu_leg):
    """Times one workload's step (attention + acceptance), and each alone;
    with ``extras`` also the paths around the step.  Returns the per-config
    record, the extra timings and what the CPU leg needs."""
    import torch
    from paper_2606_18394_amd import synth, tree_accept, tree_verify_attention
    from paper_2606_18394_amd.binding import load_library

    lib = load_library()
    w = synth.WORKLOADS[name]
    dev = torch.device("cuda:0")
    inp = synth.draw(w)
    bf = lambda a: _bf(torch, dev, a)      # noqa: E731
    i32 = lambda a: _i32(torch, dev, a)    # noqa: E731

    logits0 = torch.from_numpy(inp["logits"]).to(dev) if w.logits_dtype == "f32" \
        else bf(inp["logits"])
    # draft tokens per the workload recipe (argmax at the parent, first max)
    tgt = logits0.float().argmax(dim=-1).cpu().numpy()
    draft = synth.draft_tokens(inp["parent"], tgt, inp["match"], inp["rand_tok"])
    del tgt

    base = dict(q=bf(inp["q"]), kc=bf(inp["k_cache"]), vc=bf(inp["v_cache"]),
                kt=bf(inp["k_tree"]), vt=bf(inp["v_tree"]), logits=logits0)
    per_rep = sum(t.numel() * t.element_size() for t in base.values())
    # enough replicas that the attention-only and acceptance-only graphs, not
    # just the step, read every input from HBM
    attn_bytes, attn_flops, acc_bytes = algorithmic_work(inp, w)
    R = args.replicas or max(replicas_for(attn_bytes), replicas_for(acc_bytes))
    reuse = {"step": R * (attn_bytes + acc_bytes), "attention": R * attn_bytes,
             "accept": R * acc_bytes}
    reps = [base] + [{k: v.clone() for k, v in base.items()} for _ in range(R - 1)]
    parent, kv_len, draft_d = i32(inp["parent"]), i32(inp["kv_len"]), i32(draft)
    outs = [torch.empty(w.B, w.N, w.Hq, w.D, dtype=torch.bfloat16, device=dev) for _ in range(R)]
    acc_len = torch.empty(w.B, dtype=torch.int32, device=dev)
    path = torch.empty(w.B, w.Dmax, dtype=torch.int32, device=dev)
    targ = torch.empty(w.B, w.N, dtype=torch.int32, device=dev)
    ws_attn = torch.zeros(max(256, lib.tv_tree_verify_attention_workspace(
        w.B, w.N, w.Hq, w.Hkv, w.D, w.L)), dtype=torch.uint8, device=dev)
    ws_acc = torch.zeros(lib.tv_tree_accept_workspace(w.B, w.N, w.V), dtype=torch.uint8,
                         device=dev)

    def attn(r):
        x = reps[r]
        tree_verify_attention(x["q"], x["kc"], x["vc"], x["kt"], x["vt"], parent, outs[r],
                              kv_len=kv_len, workspace_tensor=ws_attn)

    def accept(r):
        tree_accept(reps[r]["logits"], draft_d, parent, w.Dmax, accept_len=acc_len, path=path,
                    tgt_argmax=targ, workspace_tensor=ws_acc)

    def step(r):
        attn(r)
        accept(r)

    side = torch.cuda.Stream(device=dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        for s in range(args.warmup):
            step(s % R)
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()

    timer = Timer(torch, R, args.settle_ms * 1e-3)
    for nm, fn in [("step", step), ("attn", attn), ("accept", accept)]:
        timer.capture(nm, fn)
    torch.cuda.synchronize()
    print(f"[bench] {w.name}: {R} replicas of {per_rep / 2**20:.1f} MiB; warmup done, "
          f"graphs captured", file=sys.stderr, flush=True)
    ms_step = timer.time_ms("step", args.steps)
    ms_attn = timer.time_ms("attn", args.steps)
    ms_acc = timer.time_ms("accept", args.steps)
    print(f"[bench] {w.name}: step {ms_step * 1e3:.2f} us, attention {ms_attn * 1e3:.2f} us, "
          f"accept {ms_acc * 1e3:.2f} us", file=sys.stderr, flush=True)

    # the timed graphs computed real results: keep what the oracle checks
    nodes = [check_nodes(inp["parent"][b], CHECK_NODES, 11 + b) for b in range(w.B)]
    got_all = outs[0].float().cpu().numpy()      # every replica holds the same inputs
    got_rows = [got_all[b][nodes[b]] for b in range(w.B)]
    del got_all
    acc = (acc_len.cpu().numpy(), path.cpu().numpy(), targ.cpu().numpy())

    rec = {
        "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "D": w.D, "Lmax": w.L, "N": w.N, "V": w.V,
        "logits": w.logits_dtype, "kv_len_sum": int(inp["kv_len"].sum()), "replicas": R,
        "us_per_step": ms_step * 1e3, "attention_us": ms_attn * 1e3, "accept_us": ms_acc * 1e3,
        "tree_tokens_per_s": w.B * w.N / (ms_step * 1e-3),
        "attention_bytes": attn_bytes, "attention_flops": attn_flops, "accept_bytes": acc_bytes,
        "attention_roofline": roofline("tree_verify_attention", ms_attn * 1e-3, attn_bytes,
                                       attn_flops, "attn_main", w.name),
        "accept_roofline": roofline("tree_accept", ms_acc * 1e-3, acc_bytes, 0,
                                    "accept_scan", w.name),
        "cache": cache_state(reuse),
    }

    extra = None
    if extras:
        extra = run_extras(torch, w, inp, args, dev, R, reps, parent, kv_len, draft_d, outs,
                           acc_len, path, ws_attn, attn, attn_bytes)
    cpu_in = (inp, draft, got_rows, nodes, acc) if cpu_leg else None
    del reps, outs, timer, base
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return w, rec, extra, cpu_in


def run_extras(torch, w, inp, args, dev, R, reps, parent, kv_len, draft_d, outs, acc_len, path,
               ws_attn, attn, attn_bytes):
    """The paths around the step at the headline workload, timed apart:
    drafting, the paged and tree-tail attention, the non-greedy acceptance,
    the training-mask attention, the path commit and a device-copy floor."""
    from paper_2606_18394_amd import (block_causal_attention, build_tree, commit_path,
                                      draft_topw, synth, tree_accept_sampled,
                                      tree_verify_attention, tree_verify_attention_paged)
    from paper_2606_18394_amd.binding import load_library
    lib = load_library()
    bf = lambda a: _bf(torch, dev, a)      # noqa: E731
    i32 = lambda a: _i32(torch, dev, a)    # noqa: E731

    # Tree drafting (the step that builds the verified trees): top-W of the
    # draft logits per draft depth, then the best-first tree.
    Wd = synth.draft_width(w)
    dl = synth.draft_logits(w)
    dlog0 = torch.from_numpy(dl).to(dev) if w.logits_dtype == "f32" else bf(dl)
    R_topw = replicas_for(dlog0.numel() * dlog0.element_size())   # a small input: more replicas
    dlogs = [dlog0] + [dlog0.clone() for _ in range(R_topw - 1)]
    dtok = torch.empty(w.B, w.depth, Wd, dtype=torch.int32, device=dev)
    dlp = torch.empty(w.B, w.depth, Wd, dtype=torch.float32, device=dev)
    ws_topw = torch.zeros(max(256, lib.tv_draft_topw_workspace(w.B, w.depth, w.V)),
                          dtype=torch.uint8, device=dev)

    def topw(r):
        draft_topw(dlogs[r], Wd, tok=dtok, logp=dlp, workspace_tensor=ws_topw)

    def build(r):
        build_tree(dtok, dlp, w.N)

    # The same attention over a paged cache (shuffled blocks of PAGE_BLOCK rows)
    prng = np.random.default_rng(w.seed + 77)
    mb = -(-w.L // PAGE_BLOCK)
    btab, nblk = synth.block_table(prng, w.B, mb, spare=7)
    kpool0 = bf(synth.scatter_pool(prng, inp["k_cache"], btab, nblk, PAGE_BLOCK))
    vpool0 = bf(synth.scatter_pool(prng, inp["v_cache"], btab, nblk, PAGE_BLOCK))
    pools = [(kpool0, vpool0)] + [(kpool0.clone(), vpool0.clone()) for _ in range(R - 1)]
    btab_d = i32(btab)

    def attn_paged(r):
        kp, vp = pools[r]
        x = reps[r]
        tree_verify_attention_paged(x["q"], kp, vp, btab_d, x["kt"], x["vt"], parent, outs[r],
                                    kv_len=kv_len, workspace_tensor=ws_attn)

    # tree-tail layout: the tree's K/V written into the cache after the context
    tk = np.concatenate([inp["k_cache"], np.zeros((w.B, w.N) + inp["k_cache"].shape[2:],
                                                  inp["k_cache"].dtype)], axis=1)
    tv = np.concatenate([inp["v_cache"], np.zeros_like(tk[:, :w.N])], axis=1)
    for b in range(w.B):
        kl = int(inp["kv_len"][b])
        tk[b, kl:kl + w.N] = inp["k_tree"][b]
        tv[b, kl:kl + w.N] = inp["v_tree"][b]
    tail0 = (bf(tk), bf(tv))
    tails = [tail0] + [(tail0[0].clone(), tail0[1].clone()) for _ in range(R - 1)]
    del tk, tv
    ws_tail = torch.zeros(max(256, lib.tv_tree_verify_attention_workspace(
        w.B, w.N, w.Hq, w.Hkv, w.D, w.L + w.N)), dtype=torch.uint8, device=dev)

    def attn_tail(r):
        kc, vc = tails[r]
        tree_verify_attention(reps[r]["q"], kc, vc, None, None, parent, outs[r], kv_len=kv_len,
                              workspace_tensor=ws_tail)

    # The draft head's training-mask attention at the workload's head
    # geometry: TRAIN_ANCHORS blocks of TRAIN_BLOCK positions over a
    # TRAIN_CONTEXT-row context, anchors uniform over the context.
    trng = np.random.default_rng(w.seed + 99)
    TA, TS, TL = TRAIN_ANCHORS, TRAIN_BLOCK, TRAIN_CONTEXT
    anchors_np = trng.integers(0, TL + 1, size=(1, TA)).astype(np.int32)
    tq = bf(synth._normal_bf16(trng, (1, TA, TS, w.Hq, w.D)))
    tkc = bf(synth._normal_bf16(trng, (1, TL, w.Hkv, w.D)))
    tvc = bf(synth._normal_bf16(trng, (1, TL, w.Hkv, w.D)))
    tkb = bf(synth._normal_bf16(trng, (1, TA, TS, w.Hkv, w.D)))
    tvb = bf(synth._normal_bf16(trng, (1, TA, TS, w.Hkv, w.D)))
    tanc = i32(anchors_np)
    tout = torch.empty(1, TA, TS, w.Hq, w.D, dtype=torch.bfloat16, device=dev)
    ws_train = torch.zeros(max(256, lib.tv_block_causal_attention_workspace(
        1, TA, TS, w.Hq, w.Hkv, w.D, TL)), dtype=torch.uint8, device=dev)
    train_flops = 4 * w.D * w.Hq * int(sum(int(a) * TS + TS * (TS + 1) // 2
                                           for a in anchors_np[0]))
    train_bytes = sum(t.numel() * t.element_size() for t in (tq, tkc, tvc, tkb, tvb, tout))

    def train_attn(r):
        block_causal_attention(tq, tkc, tvc, tkb, tvb, tanc, tout, workspace_tensor=ws_train)

    # committing the accepted path (kv_len is reset from a copy first, so
    # every replay commits the same rows; the reset alone is timed too and
    # subtracted)
    ccap = w.L + w.Dmax
    ckc = torch.zeros(w.B, ccap, w.Hkv, w.D, dtype=torch.bfloat16, device=dev)
    cvc = torch.zeros_like(ckc)
    ckl0 = kv_len.clone()
    ckl = kv_len.clone()

    def reset(r):
        ckl.copy_(ckl0)

    def commit(r):
        reset(r)
        commit_path(reps[r]["kt"], reps[r]["vt"], path, acc_len, ckc, cvc, ckl)

    # Non-greedy (T = 1) acceptance of the same trees: the target logits of
    # the replica, one uniform per node.
    u_acc = torch.from_numpy(np.random.default_rng(w.seed + 5).random(
        (w.B, w.N), dtype=np.float32)).to(dev)
    s_len = torch.empty(w.B, dtype=torch.int32, device=dev)
    s_path = torch.empty(w.B, w.Dmax, dtype=torch.int32, device=dev)
    s_corr = torch.empty(w.B, dtype=torch.int32, device=dev)
    ws_samp = torch.zeros(lib.tv_tree_accept_sampled_workspace(w.B, w.N, w.V),
                          dtype=torch.uint8, device=dev)

    def sampled(r):
        tree_accept_sampled(reps[r]["logits"], draft_d, parent, u_acc, 1234 + r, 1.0, w.Dmax,
                            accept_len=s_len, path=s_path, correction=s_corr,
                            workspace_tensor=ws_samp)

    # The practical floor of a streaming kernel at this size: a plain device
    # copy moving the attention's algorithmic bytes (half read, half
    # written), timed like the rest from cold replicas.
    half = max(1, attn_bytes // 4)  # int16 elements in each direction
    csrc = [torch.empty(half, dtype=torch.int16, device=dev).fill_(1) for _ in range(R)]
    cdst = [torch.empty(half, dtype=torch.int16, device=dev) for _ in range(R)]

    def copy_floor(r):
        cdst[r].copy_(csrc[r])

    for s in range(2):
        topw(s % R_topw)
        build(s % R)
        sampled(s % R)
    torch.cuda.synchronize()
    timer = Timer(torch, R, args.settle_ms * 1e-3)
    timer.capture("topw", topw, R_topw)
    for nm, fn in [("build", build), ("attn_paged", attn_paged),
                   ("attn_tail", attn_tail), ("train_attn", train_attn), ("sampled", sampled),
                   ("reset", reset), ("copy_floor", copy_floor), ("commit", commit)]:
        timer.capture(nm, fn)
    torch.cuda.synchronize()
    k = args.steps
    ms = {nm: timer.time_ms(nm, k) for nm in ["topw", "build", "attn_paged", "attn_tail",
                                              "sampled", "reset", "copy_floor", "commit"]}
    ms["train_attn"] = timer.time_ms("train_attn", max(10, k // 10))
    attn(0)
    ref0 = outs[0].clone()
    attn_paged(0)
    torch.cuda.synchronize()
    paged_same = bool(torch.equal(outs[0].view(torch.int16), ref0.view(torch.int16)))
    esz = 4 if w.logits_dtype == "f32" else 2
    # target logits read once, plus the last node's row again for the
    # correction race
    samp_bytes = (w.B * w.N + w.B) * w.V * esz
    ms_commit = max(0.0, ms["commit"] - ms["reset"])
    out = {
        "draft_topw_us": ms["topw"] * 1e3, "build_tree_us": ms["build"] * 1e3,
        "draft": {"depth": w.depth, "width": Wd, "budget": w.N},
        "paged_attention_us": ms["attn_paged"] * 1e3, "page_block": PAGE_BLOCK,
        "paged_bit_identical": paged_same,
        "tree_tail_attention_us": ms["attn_tail"] * 1e3,
        "sampled_accept": {"us": ms["sampled"] * 1e3, "temperature": 1.0, "bytes": samp_bytes,
                           "GBps": samp_bytes / (ms["sampled"] * 1e-3) / 1e9},
        "training_mask_attention": {
            "anchors": TA, "block": TS, "context": TL, "us": ms["train_attn"] * 1e3,
            "flops": train_flops, "TFLOPs": train_flops / (ms["train_attn"] * 1e-3) / 1e12,
            "mfma_frac": train_flops / (ms["train_attn"] * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
            "cache": cache_state({"training_mask_attention": train_bytes})},
        "cache": cache_state({"draft_topw": R_topw * dlog0.numel() * dlog0.element_size(),
                              "paged_attention": R * attn_bytes,
                              "tree_tail_attention": R * attn_bytes,
                              "sampled_accept": R * samp_bytes, "copy_floor": R * 4 * half}),
        "commit_us": ms_commit * 1e3, "commit_rows": int(acc_len.sum().item()),
        "copy_floor": {"bytes_moved": 4 * half, "us": ms["copy_floor"] * 1e3,
                       "GBps": 4 * half / (ms["copy_floor"] * 1e-3) / 1e9},
    }
    del timer, pools, tails, dlogs, csrc, cdst
    return out


def main():
    args = parse()
    if args.summarize_traffic:
        summarize_traffic(args.summarize_traffic, args.workload, args.kernel)
        return
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace, args.workload)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters, args.workload)
        return
    if args.copy_only:
        copy_only()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the tree-"
              f"verification path is built and timed for a single MI355X", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_18394_amd.binding import load_library

    load_library()
    torch.cuda.set_device(torch.device("cuda:0"))
    cpu_leg = not args.no_cpu_baseline and not args.core_only and \
        int(os.environ.get("RANK", "0")) == 0
    names = [args.workload] if args.core_only else \
        [args.workload] + [n for n in WORKLOAD_ORDER if n != args.workload]
    per, checks, extra, head_w, cpu = {}, {}, None, None, None
    for name in names:
        head = name == args.workload
        w, rec, ex, cpu_in = run_workload(name, args, extras=head and not args.core_only,
                                          cpu_leg=cpu_leg)
        per[name] = rec
        if head:
            extra, head_w = ex, w
        if cpu_in is not None:
            inp, draft, got_rows, nodes, acc = cpu_in
            t0 = time.perf_counter()
            checks[name] = oracle_check(inp, w, draft, got_rows, nodes, acc)
            rec["oracle_check"] = checks[name]
            print(f"[bench] {name}: oracle check {checks[name]} "
                  f"({time.perf_counter() - t0:.1f} s)", file=sys.stderr, flush=True)
            if head:
                cpu = cpu_baseline(inp, w, draft, args.cpu_budget_s)
            del inp, draft, got_rows, nodes, acc, cpu_in

    h = per[args.workload]
    w = head_w
    ms_step = h["us_per_step"] * 1e-3
    # the dominant kernel of the step: the longer of attention and acceptance
    if h["attention_us"] >= h["accept_us"]:
        roof = dict(h["attention_roofline"])
    else:
        roof = dict(h["accept_roofline"])
    detail = {"us_per_step": h["us_per_step"], "attention_us": h["attention_us"],
              "accept_us": h["accept_us"], "per_config": per}
    if extra is not None:
        detail.update(extra)
    line = {
        "metric": "tree-verify µs/step & tree-tokens/s; % of HBM/MFMA roofline at 1 MI355X",
        "value": h["tree_tokens_per_s"],
        "unit": "tree-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle_ms": args.settle_ms,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "D": w.D,
                   "Lmax": w.L, "N": w.N, "V": w.V, "logits": w.logits_dtype,
                   "kv_len_sum": h["kv_len_sum"], "replicas": h["replicas"]},
        "roofline": roof,
        "cpu_baseline": cpu,
        "detail": detail,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
