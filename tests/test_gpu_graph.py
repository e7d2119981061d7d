"""The C ABI calls captured into a HIP graph: every replay, with other eager
calls on the same workspaces between replays, gives the eager call's result
bit for bit (the split-KV counters and partials are left ready by every
call, and no call records a memset)."""
import numpy as np
import pytest
import torch

from paper_2606_18394_amd import synth
from helpers import dev_bf16, dev_i32, oracle_draft_tokens

pytestmark = pytest.mark.gpu


def _attn_inputs(w):
    inp = synth.draw(w, with_logits=False)
    return dict(q=dev_bf16(inp["q"]), kc=dev_bf16(inp["k_cache"]), vc=dev_bf16(inp["v_cache"]),
                kt=dev_bf16(inp["k_tree"]), vt=dev_bf16(inp["v_tree"]),
                par=dev_i32(inp["parent"]), kvl=dev_i32(inp["kv_len"]))


@pytest.mark.parametrize("shape", [
    dict(),                                # qwen3_8b: split KV merged inside the kernel
    dict(N=128, L=32768, depth=12),        # long context: split KV merged by a second kernel
])
def test_attention_graph_replays(shape):
    from paper_2606_18394_amd import tree_verify_attention
    from paper_2606_18394_amd.binding import load_library
    w = synth.with_shape(synth.WORKLOADS["qwen3_8b"], **shape)
    x = _attn_inputs(w)
    other = _attn_inputs(synth.with_shape(synth.WORKLOADS["qwen3_8b"], B=2, L=2048, seed=9))
    lib = load_library()
    need = max(lib.tv_tree_verify_attention_workspace(w.B, w.N, w.Hq, w.Hkv, w.D, w.L),
               lib.tv_tree_verify_attention_workspace(2, 64, w.Hq, w.Hkv, w.D, 2048))
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    out = torch.empty(w.B, w.N, w.Hq, w.D, dtype=torch.bfloat16, device="cuda")
    out2 = torch.empty(2, 64, w.Hq, w.D, dtype=torch.bfloat16, device="cuda")

    def call():
        tree_verify_attention(x["q"], x["kc"], x["vc"], x["kt"], x["vt"], x["par"], out,
                              kv_len=x["kvl"], workspace_tensor=ws)

    call()
    torch.cuda.synchronize()
    ref = out.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for rep in range(4):
        out.fill_(7.0)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), f"replay {rep}"
        # eager work of another shape on the same workspace between replays
        tree_verify_attention(other["q"], other["kc"], other["vc"], other["kt"], other["vt"],
                              other["par"], out2, kv_len=other["kvl"], workspace_tensor=ws)
        torch.cuda.synchronize()


def test_acceptance_and_drafting_graph_replays():
    from paper_2606_18394_amd import (build_tree, draft_topw, tree_accept,
                                      tree_accept_sampled)
    w = synth.with_shape(synth.WORKLOADS["qwen3_8b"], B=3, V=32000)
    inp = synth.draw(w)
    lg = dev_bf16(inp["logits"])
    draft = dev_i32(oracle_draft_tokens(inp))
    par = dev_i32(inp["parent"])
    dl = dev_bf16(synth.draft_logits(w))
    u = torch.from_numpy(np.random.default_rng(3).random((w.B, w.N), dtype=np.float32)).cuda()
    W = synth.draft_width(w)
    outs = dict(ln=torch.empty(w.B, dtype=torch.int32, device="cuda"),
                path=torch.empty(w.B, w.Dmax, dtype=torch.int32, device="cuda"),
                tgt=torch.empty(w.B, w.N, dtype=torch.int32, device="cuda"),
                sln=torch.empty(w.B, dtype=torch.int32, device="cuda"),
                spath=torch.empty(w.B, w.Dmax, dtype=torch.int32, device="cuda"),
                corr=torch.empty(w.B, dtype=torch.int32, device="cuda"),
                tok=torch.empty(w.B, w.depth, W, dtype=torch.int32, device="cuda"),
                lp=torch.empty(w.B, w.depth, W, dtype=torch.float32, device="cuda"))
    built = {}

    def call():
        tree_accept(lg, draft, par, w.Dmax, accept_len=outs["ln"], path=outs["path"],
                    tgt_argmax=outs["tgt"])
        tree_accept_sampled(lg, draft, par, u, 77, 1.0, w.Dmax, accept_len=outs["sln"],
                            path=outs["spath"], correction=outs["corr"])
        draft_topw(dl, W, tok=outs["tok"], logp=outs["lp"])
        built["t"] = build_tree(outs["tok"], outs["lp"], w.N)

    call()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in outs.items()}
    ref_tree = [t.clone() for t in built["t"]]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    # the binding allocates nothing under capture: one eager call on the
    # capturing stream creates its cached workspaces
    with torch.cuda.stream(side):
        call()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph_tree = built["t"]
    for rep in range(4):
        for v in outs.values():
            v.fill_(-5)
        for t in graph_tree:
            t.fill_(-5)
        g.replay()
        torch.cuda.synchronize()
        for k, v in outs.items():
            assert torch.equal(v, ref[k]), (k, rep)
        for a, b in zip(graph_tree, ref_tree):
            assert torch.equal(a, b), rep
        tree_accept(lg[:1].contiguous(), draft[:1].contiguous(), par[:1].contiguous(), w.Dmax)
        torch.cuda.synchronize()


def test_graph_replay_after_cached_workspace_grows():
    """A graph captured with the binding's cached workspace, then a larger
    eager call on the same stream that replaces that workspace: the replaced
    buffer stays allocated, so replays still write into memory the graph
    owns and give the eager result bit for bit."""
    from paper_2606_18394_amd import tree_verify_attention
    small = synth.WORKLOADS["qwen3_8b"]
    big = synth.with_shape(small, N=128, L=32768, depth=12)
    xs, xb = _attn_inputs(small), _attn_inputs(big)
    out = torch.empty(small.B, small.N, small.Hq, small.D, dtype=torch.bfloat16, device="cuda")
    outb = torch.empty(big.B, big.N, big.Hq, big.D, dtype=torch.bfloat16, device="cuda")

    def call(x, o):
        tree_verify_attention(x["q"], x["kc"], x["vc"], x["kt"], x["vt"], x["par"], o,
                              kv_len=x["kvl"])

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(xs, out)                      # creates the stream's cached workspace
    torch.cuda.synchronize()
    ref = out.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            call(xs, out)
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        call(xb, outb)                     # grows the cached workspace
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    filler = [torch.full((1 << 22,), 3, dtype=torch.int32, device="cuda") for _ in range(8)]
    torch.cuda.synchronize()
    for rep in range(3):
        out.fill_(7.0)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), f"replay {rep}"
        assert all(int(f.min()) == 3 and int(f.max()) == 3 for f in filler)
