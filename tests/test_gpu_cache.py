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
