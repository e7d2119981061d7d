"""GPU parity of the cache side of a verification step (App. E): attention
over a paged cache, and committing the accepted path to contiguous and paged
caches, through the C ABI.

Paged attention must give the same bits as the padded call on the gathered
cache (the same kernels read the same values), and the oracle on the gathered
cache within the attention tolerance.  Commits are bit-exact against the
oracle over whole caches and pools."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_18394_amd import synth
from helpers import dev_bf16, dev_i32, gpu_attention, oracle_attention, gpu_accept, \
    oracle_draft_tokens, host_logits_f64

pytestmark = pytest.mark.gpu
TOL = 1e-2

PAGED = [
    # (B, N, Hq, Hkv, D, block_size, max_blocks, kv_lens, spare blocks, oracle check)
    (1, 64, 32, 8, 128, 256, 16, [4000], 5, True),
    (3, 63, 8, 1, 64, 32, 40, [1280, 1, 517], 7, True),
    (4, 40, 24, 8, 128, 64, 5, [0, 300, 17, 255], 0, True),
    (2, 129, 16, 2, 128, 1024, 3, [3072, 1000], 2, False),
    (1, 64, 32, 8, 128, 128, 256, [32768], 3, False),
    (2, 17, 8, 2, 64, 32, 0, [0, 0], 0, True),
    (8, 64, 32, 4, 128, 32, 64, [2048, 1999, 33, 1024, 31, 0, 2000, 700], 11, False),
    (2, 128, 32, 4, 128, 64, 94, [5999, 1234], 3, False),
]


def _paged_inputs(case, unallocated):
    B, N, Hq, Hkv, D, bs, mb, kvl, spare, _ = PAGED[case]
    rng = np.random.default_rng(500 + case)
    trees = np.stack([synth.random_tree(rng, N, depth=min(N - 1, 12), branching=4)
                      for _ in range(B)])
    inp = synth.make_inputs(rng, B=B, N=N, Hq=Hq, Hkv=Hkv, D=D, Lmax=mb * bs, V=8,
                            trees=trees, kv_len=np.array(kvl), with_logits=False)
    used = [(k + bs - 1) // bs for k in kvl] if unallocated else None
    bt, nb = synth.block_table(rng, B, mb, spare, used)
    kp = synth.scatter_pool(rng, inp["k_cache"], bt, nb, bs)
    vp = synth.scatter_pool(rng, inp["v_cache"], bt, nb, bs)
    return inp, bt, kp, vp


def _gpu_paged(inp, bt, kp, vp):
    from paper_2606_18394_amd import tree_verify_attention_paged
    B, N, Hq, D = inp["q"].shape
    out = torch.full((B, N, Hq, D), 7.0, dtype=torch.bfloat16, device="cuda")
    tree_verify_attention_paged(dev_bf16(inp["q"]), dev_bf16(kp), dev_bf16(vp), dev_i32(bt),
                                dev_bf16(inp["k_tree"]), dev_bf16(inp["v_tree"]),
                                dev_i32(inp["parent"]), out, kv_len=dev_i32(inp["kv_len"]))
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


@pytest.mark.parametrize("unallocated", [False, True])
@pytest.mark.parametrize("case", range(len(PAGED)))
def test_paged_attention_matches_padded(case, unallocated):
    print(f"paged case {PAGED[case][:8]} unallocated={unallocated}", flush=True)
    inp, bt, kp, vp = _paged_inputs(case, unallocated)
    got = _gpu_paged(inp, bt, kp, vp)
    ref, _ = gpu_attention(inp)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
    if PAGED[case][9] and not unallocated:
        # the oracle on the cache the pool stands for, gathered by the oracle
        mb, bs = PAGED[case][6], PAGED[case][5]
        g = dict(inp)
        g["k_cache"] = oracle.gather_paged(kp, bt, mb)
        g["v_cache"] = oracle.gather_paged(vp, bt, mb)
        assert g["k_cache"].shape[1] == mb * bs
        err = np.abs(got - oracle_attention(g)).max() if got.size else 0.0
        print(f"max abs err {err:.3e}")
        assert err <= TOL


COMMIT = [
    # (B, N, Hkv, D, Lmax, Dmax)
    (1, 64, 8, 128, 4096, 9),
    (6, 40, 8, 128, 300, 7),
    (6, 63, 1, 64, 1000, 13),
    (2, 2048, 2, 128, 64, 64),
    (16, 64, 4, 128, 2048, 9),
]


def _commit_case(case):
    """Tree K/V, a path per sequence and the kv_len it lands at.  Sequence 1
    (when present) failed acceptance, sequence 2 would overflow, sequence 3
    names a node outside the tree, sequence 4 has accept_len above Dmax; the
    rest commit normally.  Also returns which sequences are valid."""
    B, N, Hkv, D, Lmax, Dmax = COMMIT[case]
    rng = np.random.default_rng(700 + case)
    kt = synth._normal_bf16(rng, (B, N, Hkv, D))
    vt = synth._normal_bf16(rng, (B, N, Hkv, D))
    n = rng.integers(1, Dmax + 1, size=B).astype(np.int32)
    path = np.full((B, Dmax), -1, np.int32)
    for b in range(B):
        path[b, 0] = 0
        path[b, 1:n[b]] = rng.integers(1, N, size=n[b] - 1) if N > 1 else 0
    kvl = rng.integers(0, Lmax - Dmax + 1, size=B).astype(np.int32)
    valid = np.ones(B, bool)
    if B > 1:
        n[1] = -1
        path[1] = -1
        valid[1] = False
    if B > 2:
        kvl[2] = Lmax - n[2] + 1
        valid[2] = False
    if B > 3:
        path[3, n[3] - 1] = N
        valid[3] = False
    if B > 4:
        n[4] = Dmax + 1
        valid[4] = False
    kvl[0] = Lmax - n[0]   # lands exactly at the capacity
    return kt, vt, path, n, kvl, valid


@pytest.mark.parametrize("case", range(len(COMMIT)))
def test_commit_contiguous(case):
    B, N, Hkv, D, Lmax, Dmax = COMMIT[case]
    print(f"commit case {COMMIT[case]}", flush=True)
    kt, vt, path, n, kvl, valid = _commit_case(case)
    rng = np.random.default_rng(900 + case)
    kc = synth._normal_bf16(rng, (B, Lmax, Hkv, D))
    vc = synth._normal_bf16(rng, (B, Lmax, Hkv, D))
    from paper_2606_18394_amd import commit_path
    dkc, dvc, dkl = dev_bf16(kc), dev_bf16(vc), dev_i32(kvl)
    commit_path(dev_bf16(kt), dev_bf16(vt), dev_i32(path), dev_i32(n), dkc, dvc, dkl)
    torch.cuda.synchronize()
    # invalid sequences are no-ops: the oracle's failed-acceptance rule
    ek, ev, el = oracle.commit_path(kc, vc, kt, vt, path, np.where(valid, n, 0), kvl)
    assert np.array_equal(dkl.cpu().numpy(), el)
    assert np.array_equal(dkc.view(torch.int16).cpu().numpy().view(np.uint16), ek)
    assert np.array_equal(dvc.view(torch.int16).cpu().numpy().view(np.uint16), ev)


@pytest.mark.parametrize("bs", [32, 256])
@pytest.mark.parametrize("case", range(len(COMMIT)))
def test_commit_paged(case, bs):
    B, N, Hkv, D, Lmax, Dmax = COMMIT[case]
    print(f"paged commit case {COMMIT[case]} block {bs}", flush=True)
    kt, vt, path, n, kvl, valid = _commit_case(case)
    rng = np.random.default_rng(950 + case)
    mb = (Lmax + bs - 1) // bs
    cap = mb * bs
    kvl = np.minimum(kvl + (cap - Lmax), cap).astype(np.int32)   # same margins to capacity
    bt, nb = synth.block_table(rng, B, mb, spare=3)
    kp = synth._normal_bf16(rng, (nb, bs, Hkv, D))
    vp = synth._normal_bf16(rng, (nb, bs, Hkv, D))
    from paper_2606_18394_amd import commit_path_paged
    dkp, dvp, dkl = dev_bf16(kp), dev_bf16(vp), dev_i32(kvl)
    commit_path_paged(dev_bf16(kt), dev_bf16(vt), dev_i32(path), dev_i32(n), dkp, dvp,
                      dev_i32(bt), dkl)
    torch.cuda.synchronize()
    ek, ev, el = oracle.commit_path_paged(kp, vp, bt, kt, vt, path, np.where(valid, n, 0), kvl,
                                          cap)
    assert np.array_equal(dkl.cpu().numpy(), el)
    assert np.array_equal(dkp.view(torch.int16).cpu().numpy().view(np.uint16), ek)
    assert np.array_equal(dvp.view(torch.int16).cpu().numpy().view(np.uint16), ev)


def test_accept_then_commit_then_attend():
    """One verification step end to end on device buffers: accept, commit the
    accepted path, and attend again over the grown cache; every stage
    against the oracle chained the same way."""
    w = synth.with_shape(synth.WORKLOADS["qwen3_8b"], B=3, V=4096, L=1024, ragged=(200, 1000))
    inp = synth.draw(w)
    Dmax = w.Dmax
    draft = oracle_draft_tokens(inp)
    ln, path, _, ok = gpu_accept(inp, draft, Dmax)
    eln, epath, _ = oracle.tree_accept(host_logits_f64(inp), draft, inp["parent"], Dmax)
    assert np.array_equal(ln, eln) and np.array_equal(path, epath)
    assert (ln >= 1).all()

    from paper_2606_18394_amd import commit_path
    kc, vc = dev_bf16(inp["k_cache"]), dev_bf16(inp["v_cache"])
    kvl = dev_i32(inp["kv_len"])
    commit_path(dev_bf16(inp["k_tree"]), dev_bf16(inp["v_tree"]), dev_i32(path), dev_i32(ln),
                kc, vc, kvl)
    torch.cuda.synchronize()
    ek, ev, el = oracle.commit_path(inp["k_cache"], inp["v_cache"], inp["k_tree"],
                                    inp["v_tree"], epath, eln, inp["kv_len"])
    assert np.array_equal(kvl.cpu().numpy(), el)
    assert np.array_equal(kc.view(torch.int16).cpu().numpy().view(np.uint16), ek)

    nxt = dict(inp)
    nxt["k_cache"], nxt["v_cache"], nxt["kv_len"] = ek, ev, el.astype(np.int32)
    got, _ = gpu_attention(nxt)
    err = np.abs(got - oracle_attention(nxt)).max()
    print(f"next-step attention max abs err {err:.3e}")
    assert err <= TOL


# ---- tree-tail layout: the tree's K/V sit in the cache right after the context

TAIL = [
    # (B, N, Hq, Hkv, D, kv_lens, extra rows past the tree, sampled oracle check)
    (1, 64, 32, 8, 128, [4000], 5, False),
    (4, 40, 24, 8, 128, [0, 31, 33, 255], 0, True),
    (3, 129, 8, 2, 64, [1, 64, 95], 7, True),
    (2, 17, 8, 1, 128, [0, 0], 0, True),
    (1, 300, 16, 2, 128, [517], 3, True),
    (8, 64, 32, 4, 128, [2048, 1999, 33, 1024, 31, 0, 2000, 700], 0, False),
    (1, 64, 32, 8, 128, [32700], 4, False),
    (2, 128, 32, 4, 128, [5900, 1234], 3, False),
]


def _tail_inputs(case):
    """Separate-tree inputs and the same data in the tree-tail layout: cache
    rows kv_len .. kv_len + N - 1 hold the tree, later rows the poison value."""
    B, N, Hq, Hkv, D, kvl, extra, _ = TAIL[case]
    rng = np.random.default_rng(800 + case)
    trees = np.stack([synth.random_tree(rng, N, depth=min(N - 1, 12), branching=4)
                      for _ in range(B)])
    Lmax = max(kvl) + N + extra
    inp = synth.make_inputs(rng, B=B, N=N, Hq=Hq, Hkv=Hkv, D=D, Lmax=Lmax, V=8, trees=trees,
                            kv_len=np.array(kvl), with_logits=False)
    kc, vc = inp["k_cache"].copy(), inp["v_cache"].copy()
    for b in range(B):
        kc[b, kvl[b]:kvl[b] + N] = inp["k_tree"][b]
        vc[b, kvl[b]:kvl[b] + N] = inp["v_tree"][b]
    return inp, kc, vc


def _gpu_tail(inp, kc, vc):
    from paper_2606_18394_amd import tree_verify_attention
    B, N, Hq, D = inp["q"].shape
    out = torch.full((B, N, Hq, D), 7.0, dtype=torch.bfloat16, device="cuda")
    tree_verify_attention(dev_bf16(inp["q"]), dev_bf16(kc), dev_bf16(vc), None, None,
                          dev_i32(inp["parent"]), out, kv_len=dev_i32(inp["kv_len"]))
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


@pytest.mark.parametrize("case", range(len(TAIL)))
def test_tree_tail_attention(case):
    print(f"tail case {TAIL[case][:6]}", flush=True)
    inp, kc, vc = _tail_inputs(case)
    got = _gpu_tail(inp, kc, vc)
    sep, _ = gpu_attention(inp)
    assert np.isfinite(got).all()
    # both within TOL of the oracle; the tilings differ, so the bf16 outputs
    # may round to neighbouring values
    assert np.abs(got - sep).max() <= 2 * TOL
    # the oracle reads the tree K/V out of the tail (the oracle's own slicing)
    g = dict(inp)
    g["k_tree"] = oracle.tree_tail(kc, inp["kv_len"], inp["N"])
    g["v_tree"] = oracle.tree_tail(vc, inp["kv_len"], inp["N"])
    B, N = inp["parent"].shape
    if TAIL[case][7]:
        ref = oracle_attention(g)
        err = np.abs(got - ref).max()
    else:
        rng = np.random.default_rng(3)
        heads = sorted(rng.choice(inp["Hq"], size=4, replace=False).tolist())
        err = 0.0
        for b in range(B):
            nodes = sorted({0, N - 1} | set(rng.choice(N, size=6, replace=False).tolist()))
            sub = {k: (v[b:b + 1] if isinstance(v, np.ndarray) and v.ndim >= 1 and
                       v.shape[0] == B else v) for k, v in g.items()}
            ref = oracle_attention(sub, nodes=nodes, heads=heads)[0]
            err = max(err, np.abs(got[b][nodes][:, heads] - ref).max())
    print(f"max abs err {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("case", [1, 2, 5])
def test_tree_tail_paged_matches_contiguous(case):
    from paper_2606_18394_amd import tree_verify_attention_paged
    inp, kc, vc = _tail_inputs(case)
    B, N, Hq, D = inp["q"].shape
    bs = 32
    mb = (kc.shape[1] + bs - 1) // bs
    pad = mb * bs - kc.shape[1]
    kc = np.concatenate([kc, np.full((B, pad) + kc.shape[2:], synth.POISON_BF16)], axis=1)
    vc = np.concatenate([vc, np.full((B, pad) + vc.shape[2:], synth.POISON_BF16)], axis=1)
    rng = np.random.default_rng(50 + case)
    bt, nb = synth.block_table(rng, B, mb, spare=5)
    kp = synth.scatter_pool(rng, kc, bt, nb, bs)
    vp = synth.scatter_pool(rng, vc, bt, nb, bs)
    out = torch.full((B, N, Hq, D), 7.0, dtype=torch.bfloat16, device="cuda")
    tree_verify_attention_paged(dev_bf16(inp["q"]), dev_bf16(kp), dev_bf16(vp), dev_i32(bt),
                                None, None, dev_i32(inp["parent"]), out,
                                kv_len=dev_i32(inp["kv_len"]))
    torch.cuda.synchronize()
    ref = _gpu_tail(inp, kc, vc)
    assert np.array_equal(out.float().cpu().numpy().view(np.uint32), ref.view(np.uint32))


def _root_paths(rng, parent, Dmax):
    """One random root-to-node path per sequence (root first), as
    tv_tree_accept writes them, and its length."""
    B, N = parent.shape
    path = np.full((B, Dmax), -1, np.int32)
    n = np.zeros(B, np.int32)
    for b in range(B):
        while True:
            u, p = int(rng.integers(0, N)), []
            while u != -1:
                p.append(u)
                u = int(parent[b, u])
            if len(p) <= Dmax:
                break
        path[b, :len(p)] = p[::-1]
        n[b] = len(p)
    return path, n


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("case", range(4))
def test_tree_tail_commit(case, paged):
    B, N, Hkv, D, Lmax, Dmax = [(1, 64, 8, 128, 4096, 13), (6, 40, 8, 128, 320, 13),
                                (5, 63, 1, 64, 960, 13), (2, 300, 2, 128, 512, 13)][case]
    print(f"tail commit case {case} paged={paged}", flush=True)
    rng = np.random.default_rng(1200 + case)
    parent = np.stack([synth.random_tree(rng, N, depth=Dmax - 1, branching=3)
                       for _ in range(B)])
    path, n = _root_paths(rng, parent, Dmax)
    kl = rng.integers(0, Lmax - N + 1, size=B).astype(np.int32)
    if B > 1:
        n[1] = -1              # failed acceptance
    if B > 2:
        kl[2] = Lmax - N + 1   # no room for the tree tail
    kl[0] = Lmax - N           # the tail ends at the capacity
    kc = synth._normal_bf16(rng, (B, Lmax, Hkv, D))
    vc = synth._normal_bf16(rng, (B, Lmax, Hkv, D))
    ek, ev, el = oracle.commit_path_tail(kc, vc, path, n, kl, N)
    from paper_2606_18394_amd import commit_path, commit_path_paged
    if not paged:
        dkc, dvc, dkl = dev_bf16(kc), dev_bf16(vc), dev_i32(kl)
        commit_path(None, None, dev_i32(path), dev_i32(n), dkc, dvc, dkl, n_nodes=N)
        torch.cuda.synchronize()
        gk, gv = dkc, dvc
    else:
        bs = 64
        mb = Lmax // bs
        assert mb * bs == Lmax
        bt, nb = synth.block_table(rng, B, mb, spare=3)
        kp = synth.scatter_pool(rng, kc, bt, nb, bs)
        vp = synth.scatter_pool(rng, vc, bt, nb, bs)
        dkp, dvp, dkl = dev_bf16(kp), dev_bf16(vp), dev_i32(kl)
        commit_path_paged(None, None, dev_i32(path), dev_i32(n), dkp, dvp, dev_i32(bt), dkl,
                          n_nodes=N)
        torch.cuda.synchronize()
        gk = torch.from_numpy(oracle.gather_paged(dkp.view(torch.int16).cpu().numpy(), bt, mb))
        gv = torch.from_numpy(oracle.gather_paged(dvp.view(torch.int16).cpu().numpy(), bt, mb))
    assert np.array_equal(dkl.cpu().numpy(), el)
    assert np.array_equal(gk.view(torch.int16).cpu().numpy().view(np.uint16), ek)
    assert np.array_equal(gv.view(torch.int16).cpu().numpy().view(np.uint16), ev)
