"""GPU parity of tree_verify_attention against the fp64 oracle (through the
C ABI).  Bar: max-abs error <= 1e-2 on bf16 N(0,1) inputs; invariances are
checked bit for bit."""
import numpy as np
import pytest
import torch

from paper_2606_18394_amd import synth
from helpers import gpu_attention, oracle_attention, oracle_attention_max_err

pytestmark = pytest.mark.gpu
TOL = 1e-2


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workload_parity(name):
    """Every output element of every workload against the fp64 oracle.  The
    oracle runs one (sequence, KV head) at a time, over that KV head's G
    query heads and all nodes, to bound its memory; together the calls
    cover every row."""
    w = synth.WORKLOADS[name]
    inp = synth.draw(w, with_logits=False)
    print(f"workload {name}: GPU attention", flush=True)
    got, ok = gpu_attention(inp, canary=4096)
    assert ok, "write outside out"
    assert np.isfinite(got).all()
    err = oracle_attention_max_err(inp, got)
    print(f"{name}: max abs err {err:.3e} over all {w.B * w.N * w.Hq} rows", flush=True)
    assert err <= TOL


FUZZ = [
    # (B, N, Hq, Hkv, D, Lmax, kv_lens, tree)
    (1, 1, 4, 4, 64, 0, [0], "random"),
    (1, 1, 8, 2, 128, 1, [1], "random"),
    (1, 2, 4, 1, 64, 63, [63], "chain"),
    (2, 3, 8, 8, 128, 64, [64, 0], "star"),
    (1, 17, 16, 2, 128, 65, [65], "random"),
    (3, 63, 8, 1, 64, 1000, [1000, 1, 517], "random"),
    (1, 64, 32, 8, 128, 64, [33], "chain"),
    (2, 65, 32, 4, 128, 1000, [999, 64], "random"),
    (1, 129, 8, 2, 64, 100, [100], "star"),
    (1, 129, 32, 8, 128, 0, [0], "random"),
    (1, 512, 16, 2, 128, 65, [65], "random"),
    (1, 512, 8, 8, 64, 16, [16], "chain"),
    (4, 40, 24, 8, 128, 300, [0, 300, 17, 255], "random"),
    (1, 2048, 2, 1, 128, 40, [40], "random"),
    (1, 300, 64, 8, 128, 2000, [1999], "random"),
    # matrix-bound shapes of several row blocks per KV head: a cache tail and
    # tree tiles after many full tiles, ragged sequences whose chunks hold 0,
    # a few or many full tiles, head dim 64
    (1, 200, 64, 8, 128, 5000, [4987], "random"),
    (3, 128, 32, 4, 128, 6000, [5999, 1234, 100], "random"),
    (1, 256, 64, 8, 64, 6000, [6000], "random"),
    (2, 128, 32, 4, 64, 6000, [6000, 37], "chain"),
    # many short ragged sequences: the longest-first ranking holds two (40
    # sequences) and eight (512 sequences) pairs per lane
    (40, 8, 8, 4, 64, 2048, [(97 * i * i + 13 * i) % 2049 for i in range(40)], "random"),
    (512, 2, 8, 8, 64, 200, [(31 * i) % 201 for i in range(512)], "random"),
]


@pytest.mark.parametrize("case", range(len(FUZZ)))
def test_fuzz_parity(case):
    B, N, Hq, Hkv, D, Lmax, kvl, kind = FUZZ[case]
    rng = np.random.default_rng(1000 + case)
    if kind == "chain":
        trees = np.stack([synth.chain_tree(N)] * B)
    elif kind == "star":
        trees = np.stack([synth.star_tree(N)] * B)
    else:
        trees = np.stack([synth.random_tree(rng, N, depth=max(1, min(N - 1, 12)), branching=4)
                          for _ in range(B)]) if N > 1 else np.full((B, 1), -1, np.int32)
    inp = synth.make_inputs(rng, B=B, N=N, Hq=Hq, Hkv=Hkv, D=D, Lmax=Lmax, V=8,
                            trees=trees, kv_len=np.array(kvl), with_logits=False)
    print(f"fuzz case {FUZZ[case]}", flush=True)
    got, ok = gpu_attention(inp, canary=1024)
    assert ok
    err = oracle_attention_max_err(inp, got)
    print(f"fuzz case {case}: max abs err {err:.3e}", flush=True)
    assert err <= TOL, err


@pytest.mark.parametrize("kvl", [0, 5, 40])
def test_zero_keys_closed_form(kvl):
    """K = 0: every visible key has the same score, so a wrong mask moves the
    output by O(1 / #visible) -- far above the tolerance at small kv_len."""
    rng = np.random.default_rng(kvl)
    B, N, Hq, Hkv, D, Lmax = 2, 200, 16, 4, 128, 64
    trees = np.stack([synth.random_tree(rng, N, depth=10, branching=3) for _ in range(B)])
    inp = synth.make_inputs(rng, B=B, N=N, Hq=Hq, Hkv=Hkv, D=D, Lmax=Lmax, V=8, trees=trees,
                            kv_len=np.array([kvl, Lmax]), with_logits=False)
    inp["k_cache"][:] = 0
    inp["k_tree"][:] = 0
    got, _ = gpu_attention(inp)
    ref = oracle_attention(inp)
    assert np.abs(got - ref).max() <= TOL


def test_masked_keys_have_no_influence():
    rng = np.random.default_rng(5)
    B, N, Hq, Hkv, D, Lmax = 1, 96, 8, 2, 128, 200
    trees = synth.random_tree(rng, N, depth=8, branching=3)[None]
    inp = synth.make_inputs(rng, B=B, N=N, Hq=Hq, Hkv=Hkv, D=D, Lmax=Lmax, V=8, trees=trees,
                            kv_len=np.array([150]), with_logits=False)
    base, _ = gpu_attention(inp)
    anc_of = []
    for i in [0, 37, N - 1]:
        anc, u = set(), i
        while u != -1:
            anc.add(u)
            u = trees[0, u]
        hidden = [u for u in range(N) if u not in anc]
        pert = dict(inp)
        for name in ["k_tree", "v_tree"]:
            arr = inp[name].copy()
            big = synth.bf16_bits(
                (np.frombuffer((arr[0, hidden].astype(np.uint32) << 16).tobytes(),
                               dtype=np.float32) * 1000).reshape(arr[0, hidden].shape))
            arr[0, hidden] = big
            pert[name] = arr
        for name in ["k_cache", "v_cache"]:
            arr = inp[name].copy()
            arr[0, 150:] = np.uint16(0x7F7F)      # huge finite values beyond kv_len
            pert[name] = arr
        got, _ = gpu_attention(pert)
        assert np.array_equal(got[0, i], base[0, i]), i


def test_deterministic_and_kvlen_default():
    w = synth.with_shape(synth.WORKLOADS["qwen3_8b"], L=1000)
    inp = synth.draw(w, with_logits=False)
    a, _ = gpu_attention(inp)
    b, _ = gpu_attention(inp)
    c, _ = gpu_attention(inp, kv_len=False)   # NULL kv_len means Lmax
    assert np.array_equal(a, b) and np.array_equal(a, c)


def test_scale_override():
    rng = np.random.default_rng(3)
    trees = synth.random_tree(rng, 20, depth=5)[None]
    inp = synth.make_inputs(rng, B=1, N=20, Hq=4, Hkv=2, D=64, Lmax=50, V=8, trees=trees,
                            kv_len=np.array([50]), with_logits=False)
    got, _ = gpu_attention(inp, scale=0.3)
    ref = oracle_attention(inp, scale=0.3)
    assert np.abs(got - ref).max() <= TOL


def test_invalid_tree_rows_are_nan():
    rng = np.random.default_rng(9)
    B, N = 3, 70
    trees = np.stack([synth.random_tree(rng, N, depth=6, branching=4) for _ in range(B)])
    trees[1, 0] = 0          # root must have parent -1
    trees[2, 40] = 45        # parent after child
    for Lmax in [64, 4000]:  # single split and split-KV paths
        inp = synth.make_inputs(rng, B=B, N=N, Hq=8, Hkv=2, D=128, Lmax=Lmax, V=8,
                                trees=trees, kv_len=np.full(B, Lmax), with_logits=False)
        got, _ = gpu_attention(inp)
        assert np.isnan(got[1]).all() and np.isnan(got[2]).all()
        ref = oracle_attention({k: (v[:1] if isinstance(v, np.ndarray) and v.ndim and
                                    v.shape[0] == B else v) for k, v in inp.items()})
        assert np.abs(got[:1] - ref).max() <= TOL


def test_workspace_reuse_across_shapes():
    """One zero-filled workspace serves calls of any sizes in any order
    (split-KV counters live at a fixed place and are left at zero): every
    result is bit-identical to the result with a fresh workspace."""
    from paper_2606_18394_amd.binding import load_library
    lib = load_library()
    ws_need = lambda w: lib.tv_tree_verify_attention_workspace(w.B, w.N, w.Hq, w.Hkv, w.D, w.L)
    W = synth.WORKLOADS
    cases = [synth.with_shape(W["long_ctx"], L=8192, N=64, depth=8),
             W["tiny"], W["qwen3_8b"],
             synth.with_shape(W["batched_30b_a3b"], B=4, L=4096),
             synth.with_shape(W["big_tree_32b"], L=2048, N=256)]
    size = max(ws_need(w) for w in cases)
    shared = torch.zeros(size, dtype=torch.uint8, device="cuda")
    inps = [synth.draw(w, with_logits=False) for w in cases]
    for rnd in range(2):
        for w, inp in zip(cases, inps):
            print(f"reuse round {rnd}: {w.name} B={w.B} N={w.N} L={w.L} ws={ws_need(w)}", flush=True)
            got, _ = gpu_attention(inp, workspace=shared)
            fresh = torch.zeros(max(256, ws_need(w)), dtype=torch.uint8, device="cuda")
            ref, _ = gpu_attention(inp, workspace=fresh)
            assert np.array_equal(got, ref), w.name
            # counters back at zero, tree flags 0 for a valid tree
            assert not fresh[:32768].any(), "sync words left non-zero"
