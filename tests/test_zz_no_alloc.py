"""The allocation-free acceptance entry point (static per-GPU scratch)
against tv_tree_accept with a workspace, through the C ABI: bit-exact on two
calls in a row, the second smaller, and on the host-detected size limit."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _case(rng, B, N, V, torch, dev, dtype):
    par = np.full((B, N), -1, dtype=np.int32)
    for b in range(B):
        for i in range(1, N):
            par[b, i] = rng.integers(0, i)
    lg = rng.normal(size=(B, N, V)).astype(np.float32)
    lg[:, :, 7] = lg.max() + 1.0          # a tie at two indices in every row
    lg[:, :, V - 3] = lg[:, :, 7]
    tgt = np.argmax(lg, axis=-1)
    tok = rng.integers(0, V, size=(B, N)).astype(np.int32)
    hit = rng.random((B, N)) < 0.6
    for b in range(B):
        for i in range(1, N):
            if hit[b, i]:
                tok[b, i] = tgt[b, par[b, i]]
    logits = torch.from_numpy(lg).to(dev).to(dtype)
    return logits, torch.from_numpy(tok).to(dev), torch.from_numpy(par).to(dev)


@pytest.mark.parametrize("dtype_name", ["bfloat16", "float32"])
def test_noalloc_matches_workspace_entry_point(dtype_name):
    from paper_2606_18394_amd import tree_accept, tree_accept_noalloc
    dev = torch.device("cuda:0")
    dtype = getattr(torch, dtype_name)
    rng = np.random.default_rng(42)
    # two calls in a row, the second with a smaller input: stale keys of the
    # first call must not leak into the second
    for B, N, V, Dmax in [(3, 300, 20011, 300), (2, 40, 5003, 40)]:
        logits, tok, par = _case(rng, B, N, V, torch, dev, dtype)
        print(f"noalloc case B={B} N={N} V={V} {dtype_name}", flush=True)
        ln = torch.full((B,), -7, dtype=torch.int32, device=dev)
        path = torch.full((B, Dmax), -7, dtype=torch.int32, device=dev)
        targ = torch.full((B, N), -7, dtype=torch.int32, device=dev)
        tree_accept_noalloc(logits, tok, par, Dmax, ln, path, targ)
        rl, rp, rt = tree_accept(logits, tok, par, Dmax)
        torch.cuda.synchronize()
        assert torch.equal(ln, rl) and torch.equal(path, rp) and torch.equal(targ, rt)
        assert (ln > 0).all()


def test_noalloc_rejects_sizes_beyond_the_scratch():
    from paper_2606_18394_amd import tree_accept_noalloc
    dev = torch.device("cuda:0")
    B, N, V = 600, 2048, 8                  # 1.2M node rows: keys exceed 8 MiB
    logits = torch.zeros(B, N, V, dtype=torch.bfloat16, device=dev)
    tok = torch.zeros(B, N, dtype=torch.int32, device=dev)
    par = torch.zeros(B, N, dtype=torch.int32, device=dev)
    ln = torch.zeros(B, dtype=torch.int32, device=dev)
    path = torch.zeros(B, 4, dtype=torch.int32, device=dev)
    with pytest.raises(RuntimeError, match="TV_ERR_SCRATCH"):
        tree_accept_noalloc(logits, tok, par, 4, ln, path)
