"""Pins of the tree-drafting oracle (Sec. 2.4 parallel tree drafting; Alg. 1):
brute-force top-W and log-softmax, a queue-free construction of best-first
expansion, closed forms (width one, full trees, breadth-first order under
equal scores) and structural invariants."""
import math

import numpy as np
import pytest

import oracle
from oracle import brute


@pytest.mark.parametrize("seed", range(4))
def test_topw_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    for V, W in [(1, 1), (5, 3), (17, 8), (40, 7)]:
        # small integers: many equal logits, ties must go to the lower index
        x = rng.integers(-3, 3, size=(3, V)).astype(np.float64)
        tok, lp = oracle.draft_topw(x, W)
        for r in range(3):
            bt, bl = brute.topw(x[r].tolist(), W)
            assert tok[r].tolist() == bt
            np.testing.assert_allclose(lp[r], bl, rtol=0, atol=1e-12)


def test_topw_closed_forms():
    # uniform logits: every log-probability is -log V
    tok, lp = oracle.draft_topw(np.full((2, 1000), 3.5), 4)
    assert tok.tolist() == [[0, 1, 2, 3]] * 2
    np.testing.assert_allclose(lp, -math.log(1000), atol=1e-12)
    # W = V: the probabilities of all tokens sum to one
    rng = np.random.default_rng(1)
    x = rng.normal(size=(4, 33)) * 5
    _, lp = oracle.draft_topw(x, 33)
    np.testing.assert_allclose(np.exp(lp).sum(-1), 1.0, atol=1e-12)
    assert (np.diff(lp, axis=-1) <= 0).all()


def _random_candidates(rng, B, Nd, W, V=1000, distinct=True):
    if distinct:
        lp = -np.sort(rng.exponential(2.0, size=(B, Nd, W)), axis=-1)  # descending, < 0
    else:
        lp = -np.sort(rng.integers(1, 4, size=(B, Nd, W)), axis=-1).astype(np.float64)
    tok = np.stack([np.stack([rng.choice(V, W, replace=False) for _ in range(Nd)])
                    for _ in range(B)])
    return tok, lp.astype(np.float32)


def _full_size(Nd, W):
    return sum(W ** d for d in range(Nd + 1))


@pytest.mark.parametrize("seed", range(8))
def test_build_matches_score_order_construction(seed):
    rng = np.random.default_rng(seed)
    for _ in range(6):
        Nd, W = int(rng.integers(1, 5)), int(rng.integers(1, 4))
        budget = int(rng.integers(1, _full_size(Nd, W) + 3))
        tok, lp = _random_candidates(rng, 2, Nd, W)
        t = oracle.build_tree(tok, lp, budget)
        for b in range(2):
            par, tk, dep, sc = brute.tree_in_score_order(tok[b].tolist(), lp[b], budget)
            n = len(par)
            assert t["n_nodes"][b] == n
            assert t["parent"][b, :n].tolist() == par
            assert t["token"][b, 1:n].tolist() == tk[1:]
            assert t["depth"][b, :n].tolist() == dep
            np.testing.assert_array_equal(t["score"][b, :n], np.array(sc, dtype=np.float32))


def test_width_one_is_a_chain():
    rng = np.random.default_rng(3)
    tok, lp = _random_candidates(rng, 1, 6, 1)
    for budget in [1, 3, 7, 20]:
        t = oracle.build_tree(tok, lp, budget)
        n = min(budget, 7)
        assert t["n_nodes"][0] == n
        assert t["parent"][0, :n].tolist() == [-1] + list(range(n - 1))
        assert t["token"][0, 1:n].tolist() == tok[0, :n - 1, 0].tolist()


@pytest.mark.parametrize("Nd,W", [(1, 4), (3, 3), (4, 2)])
def test_large_budget_gives_the_full_tree(Nd, W):
    rng = np.random.default_rng(Nd * 10 + W)
    tok, lp = _random_candidates(rng, 1, Nd, W, distinct=False)
    t = oracle.build_tree(tok, lp, _full_size(Nd, W) + 5)
    n = int(t["n_nodes"][0])
    assert n == _full_size(Nd, W)
    kids = np.bincount(t["parent"][0, 1:n], minlength=n)
    dep = t["depth"][0, :n]
    assert (kids[dep < Nd] == W).all() and (kids[dep == Nd] == 0).all()
    assert (t["token"][0, n:] == -1).all() and (t["parent"][0, n:] == -1).all()


def test_equal_scores_expand_breadth_first():
    # every candidate has log-probability -1: a node's score is -depth, ties
    # pop the lower index first, so the tree is the breadth-first prefix of
    # the full W-ary tree: parent of node i is (i - 1) // W
    W, Nd = 3, 4
    tok = np.tile(np.arange(W), (1, Nd, 1))
    lp = np.full((1, Nd, W), -1.0, dtype=np.float32)
    for budget in [2, 4, 13, 30, 40]:
        t = oracle.build_tree(tok, lp, budget)
        n = min(budget, _full_size(Nd, W))
        assert t["parent"][0, 1:n].tolist() == [(i - 1) // W for i in range(1, n)]


def test_lower_index_pops_first_on_equal_scores():
    # nodes 1 and 2 score the same; node 1 (lower index) is expanded first
    tok = np.array([[[10, 11], [20, 21]]])
    lp = np.array([[[-1.0, -1.0], [-0.5, -3.0]]], dtype=np.float32)
    t = oracle.build_tree(tok, lp, 5)
    assert t["parent"][0].tolist() == [-1, 0, 0, 1, 1]
    assert t["token"][0, 1:].tolist() == [10, 11, 20, 21]


@pytest.mark.parametrize("seed", range(4))
def test_structural_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    for distinct in [True, False]:
        Nd, W = int(rng.integers(1, 9)), int(rng.integers(1, 8))
        budget = int(rng.integers(1, 300))
        tok, lp = _random_candidates(rng, 3, Nd, W, distinct=distinct)
        root = rng.integers(0, 1000, size=3)
        t = oracle.build_tree(tok, lp, budget, root_tok=root)
        for b in range(3):
            n = int(t["n_nodes"][b])
            assert 1 <= n <= budget and t["token"][b, 0] == root[b]
            par, dep, sc = t["parent"][b], t["depth"][b], t["score"][b]
            kids = np.zeros(n, dtype=int)
            for i in range(1, n):
                p = par[i]
                assert 0 <= p < i and dep[i] == dep[p] + 1 <= Nd
                k = kids[p]
                kids[p] += 1
                assert t["token"][b, i] == tok[b, dep[p], k]     # children in candidate order
                assert sc[i] == np.float32(sc[p] + lp[b, dep[p], k])
            assert (kids <= W).all()
