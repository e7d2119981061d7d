#!/usr/bin/env python3
"""Tree-verification step benchmark on one MI355X.

A step is one pass of the whole hot path over one batch: tree-masked GQA
attention of all draft-tree nodes (one attention layer at the workload's
shape) followed by greedy tree acceptance over the nodes' target logits.
Inputs are seeded synthetic tensors of the workload's shape, resident in HBM
before timing starts; R input replicas (> 512 MB in total, twice the MI355X
last-level cache) are rotated so every step reads from HBM.

Prints one JSON line: tree-tokens/s (B*N / step time), ms per step, the
roofline position of the dominant kernel (algorithmic bytes or flops over its
event-timed duration) and the CPU oracle's throughput on a bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
MALL_BYTES = 256 << 20
PAGE_BLOCK = 64                # rows per paged-cache block in the paged timing
TRAIN_ANCHORS, TRAIN_BLOCK, TRAIN_CONTEXT = 512, 16, 4096   # training-mask attention timing


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="qwen3_8b")
    ap.add_argument("--replicas", type=int, default=0, help="0 = enough to exceed 2x the LLC")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    ap.add_argument("--copy-only", action="store_true",
                    help="only run 10 plain device copies of 256 MiB (calibrates the HBM "
                         "traffic counters: each copy reads and writes exactly 256 MiB)")
    ap.add_argument("--summarize-traffic", nargs=4, default=None,
                    metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                    help="no GPU: turn the counter CSVs of four rocprofv3 --pmc runs (FETCH_SIZE "
                         "and WRITE_SIZE of this benchmark, then of --copy-only) into "
                         "profiles/traffic_attn_main_<workload>.json and .md")
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


def summarize_traffic(dirs, workload):
    """HBM bytes per launch of the contiguous-cache attention kernel from
    FETCH_SIZE / WRITE_SIZE (KiB per dispatch), each scaled by what the same
    counter reads for a 256 MiB device copy."""
    import re
    import statistics
    # the verification launch is the contiguous-cache instantiation with the
    # most dispatches (the other timed paths launch fewer)
    pat = re.compile(r"attn_main<(\d+), (\d+), (\d+), (\d+)(?:, false)?>")
    med, names, n = {}, set(), {}
    for d, c in zip(dirs[:2], ["FETCH_SIZE", "WRITE_SIZE"]):
        by = {}
        for r in _counter_rows(d, c):
            m = pat.search(r["Kernel_Name"])
            if m:
                by.setdefault("attn_main<%s,%s,%s,%s>" % m.groups(), []).append(
                    float(r["Counter_Value"]))
        if not by:
            raise SystemExit(f"no contiguous attn_main dispatches in {d}")
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
    base = os.path.join(ROOT, "profiles", f"traffic_attn_main_{workload}")
    with open(base + ".json", "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    with open(base + ".md", "w") as fh:
        fh.write(f"""# HBM traffic: {kernel}, workload {workload}

Commands (repository root, rocprofv3 run from /tmp with TMPDIR=/tmp; one counter per run):

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d <f> -o b -- python3 bench.py --workload {workload} --no-cpu-baseline --steps 40 --warmup 5
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d <w> -o b -- python3 bench.py --workload {workload} --no-cpu-baseline --steps 40 --warmup 5
    rocprofv3 --pmc FETCH_SIZE --output-format csv -d <cf> -o c -- python3 bench.py --copy-only
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d <cw> -o c -- python3 bench.py --copy-only
    python3 bench.py --workload {workload} --summarize-traffic <f> <w> <cf> <cw>

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
    pat = re.compile(r"attn_main<(\d+), (\d+), (\d+), (\d+)(?:, false)?>")
    vals, durs, cmds = {}, {}, []
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
                     f"bench.py --workload {workload} --no-cpu-baseline --steps 20 --warmup 2")
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
    # per-dispatch durations (median, p10, p90) from the trace itself
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
    out = [f"# Kernel trace: workload {workload} (B={c['B']}, Hq={c['Hq']}, Hkv={c['Hkv']}, "
           f"D={c['D']}, L={c['Lmax']}, N={c['N']}, V={c['V']} {c['logits']})", "",
           "Command (repository root; rocprofv3 run from /tmp with TMPDIR=/tmp):", "",
           f"    rocprofv3 --kernel-trace --stats --output-format csv -d <out> -o bench -- "
           f"python3 bench.py --workload {workload} --no-cpu-baseline",
           f"    python3 bench.py --workload {workload} --summarize-trace <out> <log of the same "
           f"bench.py command without the profiler>", "",
           "Calls include warm-up, graph capture and every timed graph (step, attention, "
           "acceptance, draft top-W, tree build, paged attention, tree-tail attention, path "
           "commit).", "",
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
            f"    step {d['us_per_step']:.2f} us = attention {d['attention_us']:.2f} us + "
            f"acceptance {d['accept_us']:.2f} us",
            f"    drafting (not in the step): top-W {d['draft_topw_us']:.2f} us, tree build "
            f"{d['build_tree_us']:.2f} us",
            f"    paged attention ({d['page_block']}-row blocks) {d['paged_attention_us']:.2f} us, "
            f"tree-tail attention {d['tree_tail_attention_us']:.2f} us, "
            f"path commit {d['commit_us']:.2f} us",
            f"    non-greedy acceptance (T = 1) {d['sampled_accept']['us']:.2f} us",
            f"    training-mask attention ({d['training_mask_attention']['anchors']} blocks of "
            f"{d['training_mask_attention']['block']} over {d['training_mask_attention']['context']}"
            f" context rows) {d['training_mask_attention']['us']:.1f} us"]
    if "copy_floor" in d:
        out.append(f"    device copy of the attention's {d['copy_floor']['bytes_moved'] / 1e6:.1f} MB "
                   f"(the streaming floor) {d['copy_floor']['us']:.2f} us")
    out.append("")
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
    for f in ["tv_attention.hip", "tv_accept.hip", "tv_plan.h"]:
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


def cpu_baseline(inp, w, draft, budget_s):
    """The oracle, as it stands, on a bounded sample of the same step."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        cores = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:
        cores = 1
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
    return {"value": w.B * w.N / step, "unit": "tree-tokens/s", "cores": int(cores),
            "kind": "oracle",
            "sample": f"attention on {n_nodes}/{w.N} nodes x all {w.Hq} heads of batch {w.B} "
                      f"({t_attn:.1f} s, scaled to all nodes) + full acceptance "
                      f"({acc_step:.1f} s); fp64 numpy"}


def main():
    args = parse()
    if args.summarize_traffic:
        summarize_traffic(args.summarize_traffic, args.workload)
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
    from paper_2606_18394_amd import (block_causal_attention, build_tree, commit_path,
                                      draft_topw, synth, tree_accept, tree_accept_sampled,
                                      tree_verify_attention, tree_verify_attention_paged)
    from paper_2606_18394_amd.binding import load_library

    load_library()
    w = synth.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    inp = synth.draw(w)

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

    if w.logits_dtype == "f32":
        logits0 = torch.from_numpy(inp["logits"]).to(dev)
    else:
        logits0 = bf(inp["logits"])
    # draft tokens per the workload recipe (argmax at the parent, first max)
    tgt = logits0.float().argmax(dim=-1).cpu().numpy()
    draft = synth.draft_tokens(inp["parent"], tgt, inp["match"], inp["rand_tok"])

    base = dict(q=bf(inp["q"]), kc=bf(inp["k_cache"]), vc=bf(inp["v_cache"]),
                kt=bf(inp["k_tree"]), vt=bf(inp["v_tree"]), logits=logits0)
    per_rep = sum(t.numel() * t.element_size() for t in base.values())
    R = args.replicas or max(1, -(-2 * MALL_BYTES // per_rep))
    reps = [base] + [{k: v.clone() for k, v in base.items()} for _ in range(R - 1)]
    parent, kv_len, draft_d = i32(inp["parent"]), i32(inp["kv_len"]), i32(draft)
    outs = [torch.empty(w.B, w.N, w.Hq, w.D, dtype=torch.bfloat16, device=dev) for _ in range(R)]
    acc_len = torch.empty(w.B, dtype=torch.int32, device=dev)
    path = torch.empty(w.B, w.Dmax, dtype=torch.int32, device=dev)
    targ = torch.empty(w.B, w.N, dtype=torch.int32, device=dev)

    ws_attn = torch.zeros(
        max(256, load_library().tv_tree_verify_attention_workspace(
            w.B, w.N, w.Hq, w.Hkv, w.D, w.L)), dtype=torch.uint8, device=dev)
    ws_acc = torch.zeros(load_library().tv_tree_accept_workspace(w.B, w.N, w.V),
                         dtype=torch.uint8, device=dev)

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

    # Tree drafting (the step that builds the verified trees): top-W of the
    # draft logits per draft depth, then the best-first tree; timed apart,
    # it is not part of the verification step.
    Wd = synth.draft_width(w)
    dl = synth.draft_logits(w)
    dlog0 = torch.from_numpy(dl).to(dev) if w.logits_dtype == "f32" else bf(dl)
    dlogs = [dlog0] + [dlog0.clone() for _ in range(R - 1)]
    dtok = torch.empty(w.B, w.depth, Wd, dtype=torch.int32, device=dev)
    dlp = torch.empty(w.B, w.depth, Wd, dtype=torch.float32, device=dev)

    def topw(r):
        draft_topw(dlogs[r], Wd, tok=dtok, logp=dlp)

    # The serving side, timed apart: the same attention over a paged cache
    # (shuffled blocks of PAGE_BLOCK rows), and committing the accepted path
    # (kv_len is reset from a copy first, so every replay commits the same
    # rows; the reset alone is timed too and subtracted).
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
    kt_np, vt_np = inp["k_tree"], inp["v_tree"]
    tk = np.concatenate([inp["k_cache"], np.zeros((w.B, w.N) + inp["k_cache"].shape[2:],
                                                  inp["k_cache"].dtype)], axis=1)
    tv = np.concatenate([inp["v_cache"], np.zeros_like(tk[:, :w.N])], axis=1)
    for b in range(w.B):
        kl = int(inp["kv_len"][b])
        tk[b, kl:kl + w.N] = kt_np[b]
        tv[b, kl:kl + w.N] = vt_np[b]
    tail0 = (bf(tk), bf(tv))
    tails = [tail0] + [(tail0[0].clone(), tail0[1].clone()) for _ in range(R - 1)]
    del tk, tv

    def attn_tail(r):
        kc, vc = tails[r]
        tree_verify_attention(reps[r]["q"], kc, vc, None, None, parent, outs[r], kv_len=kv_len,
                              workspace_tensor=ws_tail)

    ws_tail = torch.zeros(
        max(256, load_library().tv_tree_verify_attention_workspace(
            w.B, w.N, w.Hq, w.Hkv, w.D, w.L + w.N)), dtype=torch.uint8, device=dev)

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
    ws_train = torch.zeros(
        max(256, load_library().tv_block_causal_attention_workspace(
            1, TA, TS, w.Hq, w.Hkv, w.D, TL)), dtype=torch.uint8, device=dev)
    train_flops = 4 * w.D * w.Hq * int(sum(int(a) * TS + TS * (TS + 1) // 2
                                           for a in anchors_np[0]))

    def train_attn(r):
        block_causal_attention(tq, tkc, tvc, tkb, tvb, tanc, tout, workspace_tensor=ws_train)

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

    def build(r):
        build_tree(dtok, dlp, w.N)

    # Non-greedy (T = 1) acceptance of the same trees: the target logits of
    # the replica, the draft head's logits, one uniform per node.
    u_acc = torch.from_numpy(np.random.default_rng(w.seed + 5).random(
        (w.B, w.N), dtype=np.float32)).to(dev)
    s_len = torch.empty(w.B, dtype=torch.int32, device=dev)
    s_path = torch.empty(w.B, w.Dmax, dtype=torch.int32, device=dev)
    s_corr = torch.empty(w.B, dtype=torch.int32, device=dev)
    ws_samp = torch.zeros(load_library().tv_tree_accept_sampled_workspace(w.B, w.N, w.V, w.depth),
                          dtype=torch.uint8, device=dev)

    def sampled(r):
        tree_accept_sampled(reps[r]["logits"], dlogs[r], draft_d, parent, u_acc, 1234 + r, 1.0,
                            w.Dmax, accept_len=s_len, path=s_path, correction=s_corr,
                            workspace_tensor=ws_samp)

    # The practical floor of a streaming kernel at this size: a plain device
    # copy moving the attention's algorithmic bytes (half read, half
    # written), timed like the rest from cold replicas.
    attn_bytes0, _, _ = algorithmic_work(inp, w)
    half = max(1, attn_bytes0 // 4)  # int16 elements in each direction
    csrc = [torch.empty(half, dtype=torch.int16, device=dev).fill_(1) for _ in range(R)]
    cdst = [torch.empty(half, dtype=torch.int16, device=dev) for _ in range(R)]

    def copy_floor(r):
        cdst[r].copy_(csrc[r])

    # Launches are recorded once into HIP graphs (one graph runs the R
    # replicas in turn, R more graphs run one replica each) so the timed
    # region measures the GPU, not Python's launch overhead.
    side = torch.cuda.Stream(device=dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        for s in range(args.warmup):
            step(s % R)
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()

    def capture(fn, rs):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for r in rs:
                fn(r)
        return g

    graphs = {}
    for s in range(2):
        topw(s % R)
        build(s % R)
    for name, fn in [("step", step), ("attn", attn), ("accept", accept), ("topw", topw),
                     ("build", build), ("attn_paged", attn_paged), ("attn_tail", attn_tail),
                     ("train_attn", train_attn), ("sampled", sampled),
                     ("reset", reset), ("copy_floor", copy_floor),
                     ("commit", commit)]:
        graphs[name] = (capture(fn, range(R)), [capture(fn, [r]) for r in range(R)])
    torch.cuda.synchronize()
    print(f"[bench] {w.name}: {R} replicas of {per_rep / 2**20:.1f} MiB; warmup done, "
          f"graphs captured", file=sys.stderr, flush=True)

    def timed(name, k):
        full, singles = graphs[name]
        for _ in range(2):             # untimed graph warmup
            full.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(k // R):
            full.replay()
        for r in range(k % R):
            singles[r].replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / k     # ms

    ms_step = timed("step", args.steps)
    ms_attn = timed("attn", args.steps)
    ms_acc = timed("accept", args.steps)
    ms_topw = timed("topw", args.steps)
    ms_build = timed("build", args.steps)
    ms_paged = timed("attn_paged", args.steps)
    ms_tail = timed("attn_tail", args.steps)
    ms_train = timed("train_attn", max(10, args.steps // 10))
    ms_samp = timed("sampled", args.steps)
    ms_commit = max(0.0, timed("commit", args.steps) - timed("reset", args.steps))
    ms_copy = timed("copy_floor", args.steps)
    attn(0)
    ref0 = outs[0].clone()
    attn_paged(0)
    torch.cuda.synchronize()
    paged_same = bool(torch.equal(outs[0].view(torch.int16), ref0.view(torch.int16)))
    print(f"[bench] step {ms_step * 1e3:.2f} us, attention {ms_attn * 1e3:.2f} us, "
          f"accept {ms_acc * 1e3:.2f} us", file=sys.stderr, flush=True)

    # the graphs computed real results: check the last accept against the
    # oracle-free expectation that the path is a valid root chain
    ln = int(acc_len[0].item())
    assert 1 <= ln <= w.Dmax, ln

    attn_bytes, attn_flops, acc_bytes = algorithmic_work(inp, w)
    # target logits + draft logits read once, plus two rows per sequence for
    # the correction race
    esz = 4 if w.logits_dtype == "f32" else 2
    samp_bytes = (w.B * (w.N + w.depth) + 2 * w.B) * w.V * esz
    if ms_attn >= ms_acc:
        t = ms_attn * 1e-3
        if attn_bytes / (HBM_PEAK_GBS * 1e9) >= attn_flops / (BF16_PEAK_TFLOPS * 1e12):
            roof = {"bound": "hbm", "achieved": attn_bytes / t / 1e9, "peak": HBM_PEAK_GBS,
                    "unit": "GB/s"}
        else:
            roof = {"bound": "mfma", "achieved": attn_flops / t / 1e12,
                    "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
        roof["kernel"] = "tree_verify_attention"
        roof["traffic"] = measured_traffic("attn_main", w.name)
    else:
        t = ms_acc * 1e-3
        roof = {"bound": "hbm", "achieved": acc_bytes / t / 1e9, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "kernel": "tree_accept",
                "traffic": measured_traffic("accept_scan", w.name)}
    roof["frac"] = roof["achieved"] / roof["peak"]

    cpu = None
    if not args.no_cpu_baseline and int(os.environ.get("RANK", "0")) == 0:
        cpu = cpu_baseline(inp, w, draft, args.cpu_budget_s)

    tokens = w.B * w.N
    line = {
        "metric": "tree-verify \u00b5s/step & tree-tokens/s; % of HBM/MFMA roofline at 1 MI355X",
        "value": tokens / (ms_step * 1e-3),
        "unit": "tree-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "D": w.D,
                   "Lmax": w.L, "N": w.N, "V": w.V, "logits": w.logits_dtype,
                   "kv_len_sum": int(inp["kv_len"].sum()), "replicas": R},
        "roofline": roof,
        "cpu_baseline": cpu,
        "detail": {"us_per_step": ms_step * 1e3, "attention_us": ms_attn * 1e3,
                   "accept_us": ms_acc * 1e3, "attention_bytes": attn_bytes,
                   "attention_flops": attn_flops, "accept_bytes": acc_bytes,
                   "attention_GBps": attn_bytes / (ms_attn * 1e-3) / 1e9,
                   "attention_TFLOPs": attn_flops / (ms_attn * 1e-3) / 1e12,
                   "accept_GBps": acc_bytes / (ms_acc * 1e-3) / 1e9,
                   "draft_topw_us": ms_topw * 1e3, "build_tree_us": ms_build * 1e3,
                   "draft": {"depth": w.depth, "width": Wd, "budget": w.N},
                   "paged_attention_us": ms_paged * 1e3, "page_block": PAGE_BLOCK,
                   "paged_bit_identical": paged_same,
                   "paged_attention_GBps": attn_bytes / (ms_paged * 1e-3) / 1e9,
                   "tree_tail_attention_us": ms_tail * 1e3,
                   "sampled_accept": {
                       "us": ms_samp * 1e3, "temperature": 1.0,
                       "bytes": samp_bytes, "GBps": samp_bytes / (ms_samp * 1e-3) / 1e9},
                   "training_mask_attention": {
                       "anchors": TA, "block": TS, "context": TL, "us": ms_train * 1e3,
                       "flops": train_flops,
                       "TFLOPs": train_flops / (ms_train * 1e-3) / 1e12,
                       "mfma_frac": train_flops / (ms_train * 1e-3) / 1e12 / BF16_PEAK_TFLOPS},
                   "commit_us": ms_commit * 1e3, "commit_rows": int(acc_len.sum().item()),
                   "copy_floor": {"bytes_moved": 4 * half, "us": ms_copy * 1e3,
                                  "GBps": 4 * half / (ms_copy * 1e-3) / 1e9}},
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
