"""GPU parity of tree_accept against the oracle: bit-exact accept_len, path
and per-node argmax (through the C ABI)."""
import numpy as np
import pytest

import oracle
from paper_2606_18394_amd import synth
from helpers import gpu_accept, host_logits_f64, oracle_draft_tokens

pytestmark = pytest.mark.gpu


def _compare(inp, draft, Dmax, canary=0, workspace=None):
    ln, path, tgt, ok = gpu_accept(inp, draft, Dmax, canary=canary, workspace=workspace)
    rl, rp, rt = oracle.tree_accept(host_logits_f64(inp), draft, inp["parent"], Dmax)
    np.testing.assert_array_equal(tgt, rt)
    np.testing.assert_array_equal(ln, rl)
    np.testing.assert_array_equal(path, rp)
    assert ok, "write outside the outputs"
    return ln


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workload_parity(name):
    w = synth.WORKLOADS[name]
    inp = synth.draw(w)
    draft = oracle_draft_tokens(inp)
    ln = _compare(inp, draft, w.Dmax, canary=256)
    print(f"{name}: accept_len {ln.tolist()[:16]}")
    # second call on the same workspace (tickets must have been reset)
    _compare(inp, draft, w.Dmax)


def _small(rng, B, N, V, dtype, depth=6, width=3):
    trees = np.stack([synth.random_tree(rng, N, depth=min(depth, N - 1) if N > 1 else 1,
                                        branching=width) if N > 1 else
                      np.array([-1], np.int32) for _ in range(B)])
    inp = synth.make_inputs(rng, B=B, N=N, Hq=1, Hkv=1, D=8, Lmax=1, V=V, trees=trees,
                            kv_len=np.ones(B), logits_dtype=dtype, p_match=0.7)
    return inp


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("V", [1, 3, 8, 1000, 1001, 4099, 151936])
def test_vocab_sizes(dtype, V):
    rng = np.random.default_rng(V)
    inp = _small(rng, 3, 33, V, dtype)
    _compare(inp, oracle_draft_tokens(inp), 8, canary=64)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_tie_stress(dtype):
    rng = np.random.default_rng(1)
    B, N, V = 2, 48, 5000
    inp = _small(rng, B, N, V, dtype)
    lg = host_logits_f64(inp)
    lg[0, 0, :] = 1.0                       # constant row -> index 0
    lg[0, 1, [0, V - 1]] = 50.0             # maxima at both ends
    lg[0, 2, :] = -3.0
    lg[0, 2, [17, 4000]] = [-0.0, 0.0]      # -0.0 before +0.0: tie, index 17
    lg[0, 3, :] = -3.0
    lg[0, 3, [17, 4000]] = [0.0, -0.0]
    lg[1, :, :] = np.round(lg[1] * 2) / 2   # coarse values: many ties
    lg[1, 5, :] = -np.inf
    lg[1, 6, 123] = np.inf
    if dtype == "bf16":
        inp["logits"] = synth.bf16_bits(lg.astype(np.float32))
    else:
        inp["logits"] = lg.astype(np.float32)
    _compare(inp, oracle_draft_tokens(inp), 7)


def test_duplicate_siblings_and_full_match():
    rng = np.random.default_rng(2)
    inp = _small(rng, 4, 100, 50, "bf16", depth=8, width=4)
    tgt = oracle.target_argmax(host_logits_f64(inp))
    full = synth.draft_tokens(inp["parent"], tgt, np.ones((4, 100), bool), inp["rand_tok"])
    ln = _compare(inp, full, 9)
    none = (full + 1) % 50
    none[:, 0] = 0
    ln0 = _compare(inp, none, 9)
    assert (ln0 == 1).all() and (ln >= 1).all()


def test_errors_and_short_dmax():
    rng = np.random.default_rng(4)
    inp = _small(rng, 4, 30, 64, "bf16", depth=5)
    inp["parent"][1, 0] = 3
    inp["parent"][2, 7] = 9
    draft = oracle_draft_tokens(inp)
    for Dmax in [1, 2, 6, 40]:
        ln = _compare(inp, draft, Dmax)
        assert ln[1] == -1 and ln[2] == -1


def test_many_sequences_single_node():
    rng = np.random.default_rng(5)
    inp = _small(rng, 300, 1, 777, "f32")
    ln = _compare(inp, oracle_draft_tokens(inp), 1)
    assert (ln == 1).all()


def test_max_nodes_chain():
    rng = np.random.default_rng(6)
    N = 2048
    trees = synth.chain_tree(N)[None]
    inp = synth.make_inputs(rng, B=1, N=N, Hq=1, Hkv=1, D=8, Lmax=1, V=40, trees=trees,
                            kv_len=np.ones(1), logits_dtype="bf16", p_match=0.995)
    draft = oracle_draft_tokens(inp)
    _compare(inp, draft, N)
    _compare(inp, draft, 10)


def test_workspace_reuse_across_shapes():
    """One workspace serves calls of different shapes back to back, with
    exact results every time."""
    import torch
    from paper_2606_18394_amd.binding import load_library
    lib = load_library()
    rng = np.random.default_rng(8)
    shapes = [(16, 64, 3000, "bf16"), (300, 1, 777, "f32"), (2, 500, 9000, "bf16"),
              (40, 7, 5, "f32"), (100, 3, 50, "bf16"), (16, 64, 3000, "bf16")]
    size = max(lib.tv_tree_accept_workspace(B, N, V) for B, N, V, _ in shapes)
    ws = torch.zeros(size, dtype=torch.uint8, device="cuda")
    for B, N, V, dt in shapes:
        inp = _small(rng, B, N, V, dt)
        print(f"accept reuse B={B} N={N} V={V} {dt}", flush=True)
        _compare(inp, oracle_draft_tokens(inp), 6, workspace=ws)


@pytest.mark.parametrize("B", [8, 9])
def test_row_count_plans(B):
    """Many sequences of the largest tree: the per-sequence workgroups
    each merge 2048 rows of split keys."""
    rng = np.random.default_rng(20 + B)
    inp = _small(rng, B, 2048, 48, "bf16", depth=14, width=4)
    _compare(inp, oracle_draft_tokens(inp), 16)


@pytest.mark.parametrize("N", [65, 100, 128, 129, 200, 256, 257, 300, 511, 512, 513])
def test_node_counts_around_the_one_wave_limits(N):
    """Trees whose nodes share a wave's lanes (one to eight per lane) and
    the first size past them; bushy random trees, a full chain, and an
    invalid parent in a later lane slot."""
    rng = np.random.default_rng(300 + N)
    B = 3
    inp = _small(rng, B, N, 700, "bf16", depth=min(20, N - 1), width=6)
    inp["parent"][1] = synth.chain_tree(N)
    draft = oracle_draft_tokens(inp)
    tgt = oracle.target_argmax(host_logits_f64(inp))
    draft[1, 1:] = tgt[1, :-1]              # the chain is accepted end to end
    ln = _compare(inp, draft, N)
    assert ln[1] == N
    _compare(inp, draft, 12)                 # the chain's path is too long: sentinel
    inp["parent"][2, N - 1] = N - 1          # invalid: a node its own parent
    ln = _compare(inp, draft, N)
    assert ln[2] == -1


@pytest.mark.parametrize("N", [129, 300])
def test_finish_with_most_split_keys(N):
    """One sequence over a large f32 vocabulary: the most vocabulary splits
    the plan gives (16 at 129 nodes), so the finish of trees over 128 nodes
    merges its largest number of split keys per node."""
    rng = np.random.default_rng(700 + N)
    inp = _small(rng, 1, N, 151936, "f32", depth=12, width=5)
    _compare(inp, oracle_draft_tokens(inp), 16)
