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
    return ap.parse_args()


COPY_BYTES = 256 << 20


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
    if args.copy_only:
        copy_only()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the tree-"
              f"verification path is built and timed for a single MI355X", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_18394_amd import build_tree, draft_topw, synth, tree_accept, tree_verify_attention
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

    def build(r):
        build_tree(dtok, dlp, w.N)

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
                     ("build", build)]:
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
    print(f"[bench] step {ms_step * 1e3:.2f} us, attention {ms_attn * 1e3:.2f} us, "
          f"accept {ms_acc * 1e3:.2f} us", file=sys.stderr, flush=True)

    # the graphs computed real results: check the last accept against the
    # oracle-free expectation that the path is a valid root chain
    ln = int(acc_len[0].item())
    assert 1 <= ln <= w.Dmax, ln

    attn_bytes, attn_flops, acc_bytes = algorithmic_work(inp, w)
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
                   "draft": {"depth": w.depth, "width": Wd, "budget": w.N}},
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
