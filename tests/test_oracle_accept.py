"""Pins of the acceptance oracle (Sec. 2.4 greedy rule; App. E): explicit
path enumeration, constructed special cases, argmax tie rules, the error
sentinels, and the expected-tokens closed form of Sec. 2.1 on chain trees."""
import numpy as np
import pytest

import oracle
from oracle import brute
from paper_2606_18394_amd import synth


def _check_against_brute(logits, draft, parent, Dmax):
    ln, path, tgt = oracle.tree_accept(logits, draft, parent, Dmax)
    bl, bp, bt = brute.accept(logits.tolist(), draft.tolist(), parent.tolist(), Dmax)
    np.testing.assert_array_equal(tgt, np.array(bt))
    np.testing.assert_array_equal(ln, np.array(bl))
    np.testing.assert_array_equal(path, np.array(bp))
    return ln, path, tgt


def _feasible_tree(rng, N):
    depth, width = int(rng.integers(1, 6)), int(rng.integers(1, 4))
    try:
        return synth.random_tree(rng, N, depth=depth, branching=width)
    except ValueError:          # caps too tight for N nodes
        return synth.random_tree(rng, N, depth=depth)


@pytest.mark.parametrize("seed", range(6))
def test_matches_path_enumeration(seed):
    rng = np.random.default_rng(seed)
    B, V = 8, 5
    for N in [1, 2, 7, 20]:
        trees = np.stack([_feasible_tree(rng, N) for _ in range(B)])
        # small integer logits: frequent ties and frequent matches
        logits = rng.integers(-2, 3, size=(B, N, V)).astype(np.float64)
        tgt = oracle.target_argmax(logits)
        draft = synth.draft_tokens(trees, tgt, rng.random((B, N)) < 0.7,
                                   rng.integers(0, V, size=(B, N)))
        for Dmax in [1, 3, 8]:
            _check_against_brute(logits, draft, trees, Dmax)


def test_all_match_takes_lowest_index_deepest_node():
    parent = np.array([[-1, 0, 0, 1, 2, 2, 3, 4]])
    # depths:           0  1  1  2  2  2  3  3  -> deepest nodes 6 and 7
    rng = np.random.default_rng(0)
    logits = rng.standard_normal((1, 8, 10))
    tgt = oracle.target_argmax(logits)
    draft = np.array([[0] + [tgt[0, parent[0, i]] for i in range(1, 8)]])
    ln, path, _ = _check_against_brute(logits, draft, parent, 6)
    assert ln[0] == 4
    assert path[0].tolist() == [0, 1, 3, 6, -1, -1]


def test_no_match_accepts_root_only():
    parent = np.array([[-1, 0, 1, 2, 0]])
    logits = np.zeros((1, 5, 4))
    logits[:, :, 2] = 1.0            # argmax 2 everywhere
    draft = np.array([[2, 0, 1, 3, 3]])
    ln, path, tgt = _check_against_brute(logits, draft, parent, 4)
    assert ln[0] == 1 and path[0].tolist() == [0, -1, -1, -1]
    assert (tgt == 2).all()


def test_root_token_is_ignored():
    parent = np.array([[-1, 0]])
    logits = np.zeros((1, 2, 3))
    logits[0, 0, 1] = 5.0
    for root_tok in [0, 1, 2, 999]:
        ln, path, _ = oracle.tree_accept(logits, np.array([[root_tok, 1]]), parent, 2)
        assert ln[0] == 2 and path[0].tolist() == [0, 1]


def test_argmax_ties_lowest_index_and_signed_zero():
    lg = np.full((1, 3, 9), -1.0)
    lg[0, 0, [3, 7]] = 2.5                  # duplicated maximum
    lg[0, 1, 2] = -0.0                      # -0.0 before +0.0: equal values
    lg[0, 1, 5] = 0.0
    lg[0, 2, :] = 4.0                       # constant row
    tgt = oracle.target_argmax(lg)
    assert tgt.tolist() == [[3, 2, 0]]
    assert [brute.argmax_first(r) for r in lg[0].tolist()] == [3, 2, 0]
    lg[0, 1, 2], lg[0, 1, 5] = 0.0, -0.0
    assert oracle.target_argmax(lg)[0, 1] == 2


def test_equal_depth_accepted_nodes_pick_lowest_index():
    # duplicate sibling tokens: nodes 1 and 2 both match, 3 (child of 2) and
    # 4 (child of 1) both match -> depth 2 tie, lowest index is 3
    parent = np.array([[-1, 0, 0, 2, 1]])
    logits = np.zeros((1, 5, 4))
    logits[0, :, 1] = 1.0
    draft = np.array([[0, 1, 1, 1, 1]])
    ln, path, _ = _check_against_brute(logits, draft, parent, 5)
    assert ln[0] == 3 and path[0, :3].tolist() == [0, 2, 3]


def test_error_sentinels():
    logits = np.zeros((3, 4, 3))
    logits[:, :, 0] = 1
    draft = np.zeros((3, 4), dtype=np.int64)
    parent = np.array([[-1, 0, 1, 2], [-1, 0, 2, 1], [0, 0, 1, 2]])
    ln, path, tgt = _check_against_brute(logits, draft, parent, 3)
    # seq 0: chain of depth 3 fully accepted needs 4 entries > Dmax=3
    assert ln.tolist() == [-1, -1, -1]
    assert (path == -1).all()
    assert (tgt == 0).all()
    ln, path, _ = oracle.tree_accept(logits, draft, parent, 4)
    assert ln.tolist() == [4, -1, -1] and path[0].tolist() == [0, 1, 2, 3]


def test_chain_mean_accept_len_matches_expected_tokens_formula():
    """Sec. 2.1: with i.i.d. per-token acceptance alpha and n drafts, the
    expected tokens per step is (1 - alpha^(n+1)) / (1 - alpha).  A chain of
    N nodes has n = N - 1 drafts and accept_len = accepted drafts + 1.  A
    draft copies the target argmax with probability p, otherwise it is uniform
    over V and still matches with probability 1/V."""
    rng = np.random.default_rng(2024)
    M, N, V, p = 20000, 6, 8, 0.5
    alpha = p + (1 - p) / V
    parent = np.stack([synth.chain_tree(N)] * M)
    logits = rng.standard_normal((M, N, V))
    tgt = oracle.target_argmax(logits)
    draft = synth.draft_tokens(parent, tgt, rng.random((M, N)) < p,
                               rng.integers(0, V, size=(M, N)))
    ln, _, _ = oracle.tree_accept(logits, draft, parent, N)
    expect = (1 - alpha ** N) / (1 - alpha)
    sem = ln.std() / np.sqrt(M)
    assert abs(ln.mean() - expect) < 5 * sem, (ln.mean(), expect, sem)
    # the geometric law itself: P(accept_len >= r + 1) = alpha^r
    for r in range(1, N):
        frac = (ln >= r + 1).mean()
        assert abs(frac - alpha ** r) < 5 * np.sqrt(alpha ** r * (1 - alpha ** r) / M)


def test_path_is_a_root_chain():
    rng = np.random.default_rng(3)
    B, N, V = 16, 30, 3
    trees = np.stack([synth.random_tree(rng, N, depth=8, branching=4) for _ in range(B)])
    logits = rng.standard_normal((B, N, V))
    tgt = oracle.target_argmax(logits)
    draft = synth.draft_tokens(trees, tgt, rng.random((B, N)) < 0.8, rng.integers(0, V, (B, N)))
    ln, path, _ = oracle.tree_accept(logits, draft, trees, 9)
    for b in range(B):
        p = path[b, :ln[b]]
        assert p[0] == 0 and (path[b, ln[b]:] == -1).all()
        for t in range(1, ln[b]):
            assert trees[b, p[t]] == p[t - 1]
            assert draft[b, p[t]] == tgt[b, p[t - 1]]
