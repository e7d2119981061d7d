"""Shared test plumbing: move synthetic inputs to the GPU, call the HIP path
through the C ABI binding, and evaluate the oracle on the same inputs."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2606_18394_amd import synth


def dev_bf16(bits: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(
        torch.bfloat16).to(device)


def dev_i32(x: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(device)


def dev_logits(inp: dict, device="cuda") -> torch.Tensor:
    if inp["logits_dtype"] == "f32":
        return torch.from_numpy(np.ascontiguousarray(inp["logits"])).to(device)
    return dev_bf16(inp["logits"], device)


def host_logits_f64(inp: dict) -> np.ndarray:
    if inp["logits_dtype"] == "f32":
        return inp["logits"].astype(np.float64)
    return oracle.decode_bf16(inp["logits"])


def gpu_attention(inp: dict, scale=None, kv_len=True, canary: int = 0, workspace=None):
    """Runs the HIP attention; returns (out fp32 numpy [B,N,Hq,D], canary_ok)."""
    from paper_2606_18394_amd import tree_verify_attention
    B, N, Hq, D = inp["q"].shape
    n = B * N * Hq * D
    buf = torch.full((n + 2 * canary,), 7.0, dtype=torch.bfloat16, device="cuda")
    out = buf[canary:canary + n].view(B, N, Hq, D)
    tree_verify_attention(dev_bf16(inp["q"]), dev_bf16(inp["k_cache"]),
                          dev_bf16(inp["v_cache"]), dev_bf16(inp["k_tree"]),
                          dev_bf16(inp["v_tree"]), dev_i32(inp["parent"]), out,
                          kv_len=dev_i32(inp["kv_len"]) if kv_len else None, scale=scale,
                          workspace_tensor=workspace)
    torch.cuda.synchronize()
    ok = True
    if canary:
        ok = bool((buf[:canary] == 7.0).all() and (buf[canary + n:] == 7.0).all())
    return out.float().cpu().numpy(), ok


def oracle_attention(inp: dict, nodes=None, heads=None, scale=None):
    return oracle.tree_attention(
        oracle.decode_bf16(inp["q"]), oracle.decode_bf16(inp["k_cache"]),
        oracle.decode_bf16(inp["v_cache"]), oracle.decode_bf16(inp["k_tree"]),
        oracle.decode_bf16(inp["v_tree"]), inp["parent"], inp["kv_len"],
        scale=scale, nodes=nodes, heads=heads)


def oracle_draft_tokens(inp: dict) -> np.ndarray:
    """Draft tokens as the workload recipe defines them, using the oracle's
    argmax at the parent."""
    tgt = oracle.target_argmax(host_logits_f64(inp))
    return synth.draft_tokens(inp["parent"], tgt, inp["match"], inp["rand_tok"])


def gpu_accept(inp: dict, draft: np.ndarray, Dmax: int, canary: int = 0, workspace=None):
    from paper_2606_18394_amd import tree_accept
    B, N = inp["parent"].shape
    lbuf = torch.full((B + 2 * canary,), -77, dtype=torch.int32, device="cuda")
    pbuf = torch.full((B * Dmax + 2 * canary,), -77, dtype=torch.int32, device="cuda")
    tbuf = torch.full((B * N + 2 * canary,), -77, dtype=torch.int32, device="cuda")
    ln = lbuf[canary:canary + B]
    path = pbuf[canary:canary + B * Dmax].view(B, Dmax)
    tgt = tbuf[canary:canary + B * N].view(B, N)
    tree_accept(dev_logits(inp), dev_i32(draft), dev_i32(inp["parent"]), Dmax,
                accept_len=ln, path=path, tgt_argmax=tgt, workspace_tensor=workspace)
    torch.cuda.synchronize()
    ok = True
    if canary:
        for buf, n in [(lbuf, B), (pbuf, B * Dmax), (tbuf, B * N)]:
            ok &= bool((buf[:canary] == -77).all() and (buf[canary + n:] == -77).all())
    return ln.cpu().numpy(), path.cpu().numpy(), tgt.cpu().numpy(), ok


def oracle_attention_max_err(inp: dict, got: np.ndarray, scale=None) -> float:
    """Max-abs difference between ``got`` [B,N,Hq,D] and the oracle over every
    output element.  The oracle runs one (sequence, KV head) at a time, over
    that head's G query heads and all nodes, which bounds its memory; the
    calls together cover every row."""
    B, N, Hq, D = inp["q"].shape
    Hkv = inp["k_cache"].shape[2]
    G = Hq // Hkv
    dec = oracle.decode_bf16
    err = 0.0
    for b in range(B):
        sl = slice(b, b + 1)
        q, kt, vt = dec(inp["q"][sl]), dec(inp["k_tree"][sl]), dec(inp["v_tree"][sl])
        kc, vc = dec(inp["k_cache"][sl]), dec(inp["v_cache"][sl])
        for g in range(Hkv):
            heads = np.arange(g * G, (g + 1) * G)
            ref = oracle.tree_attention(q, kc, vc, kt, vt, inp["parent"][sl], inp["kv_len"][sl],
                                        scale=scale, heads=heads)[0]
            d = np.abs(got[b][:, heads] - ref)
            if np.isnan(ref).all():
                if not np.isnan(got[b]).all():
                    return float("inf")
                continue
            err = max(err, float(d.max()))
    return err
