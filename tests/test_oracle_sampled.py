"""Pins of the non-greedy tree-acceptance oracle (Sec. 2.4 speculative
sampling rule applied to each node's deterministic children against the
target's residual, correction from the final residual; lossless as Sec. 2.2
states) and of its counter-based generator."""
import os

import numpy as np
import pytest

from oracle import brute, tree_accept
from oracle.philox import philox4x32, philox4x32_array, uniform_open
from oracle.tree_accept_sampled import race_sample, tree_accept_sampled

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat():
    rows = []
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        w = [int(x, 16) for x in line.split()]
        rows.append((w[:4], w[4:6], w[6:]))
    return rows


def test_philox_known_answers():
    rows = _kat()
    assert len(rows) == 3
    for ctr, key, out in rows:
        assert list(philox4x32(ctr, key)) == out
        arr = philox4x32_array(*[np.array([c]) for c in ctr], key[0], key[1])
        assert [int(a[0]) for a in arr] == out


def test_philox_array_matches_scalar():
    rng = np.random.default_rng(0)
    ctr = rng.integers(0, 2**32, size=(50, 4), dtype=np.uint64)
    key = (0x12345678, 0x9ABCDEF0)
    arr = philox4x32_array(ctr[:, 0], ctr[:, 1], ctr[:, 2], ctr[:, 3], *key)
    for n in range(50):
        assert tuple(int(a[n]) for a in arr) == philox4x32(ctr[n], key)


def test_uniform_is_open_and_exact_in_fp32():
    assert uniform_open(0) == 0.5 / 2**23
    assert uniform_open(0xFFFFFFFF) == 1 - 0.5 / 2**23
    assert 0 < uniform_open(0) < uniform_open(0xFFFFFFFF) < 1
    rng = np.random.default_rng(1)
    for w in rng.integers(0, 2**32, size=1000):
        u = uniform_open(int(w))
        assert float(np.float32(u)) == u


def _case(rng, B=3, N=10, V=6, depth=4, dup=True):
    par = np.zeros((B, N), dtype=int)
    for b in range(B):
        par[b, 0] = -1
        dep = [0]
        for i in range(1, N):
            cand = [j for j in range(i) if dep[j] < depth]
            par[b, i] = rng.choice(cand)
            dep.append(dep[par[b, i]] + 1)
    lg = rng.normal(size=(B, N, V)) * 1.5
    tok = rng.integers(0, V, size=(B, N))
    if not dup:      # distinct tokens among every node's children
        for b in range(B):
            for v in range(N):
                kids = [c for c in range(1, N) if par[b, c] == v]
                tok[b, kids] = rng.permutation(V)[:len(kids)]
    u = rng.random((B, N))
    return lg, tok, par, u


@pytest.mark.parametrize("seed", range(10))
def test_matches_path_enumeration(seed):
    rng = np.random.default_rng(seed)
    lg, tok, par, u = _case(rng, V=5 if seed % 2 else 7)
    if seed == 3:
        tok[0, 4] = -2          # a token outside the vocabulary never passes
        tok[1, 2] = 99
    T = [1.0, 0.7, 1.6][seed % 3]
    got = tree_accept_sampled(lg, tok, par, u, 1000 + seed, T, 6, detail=True)
    assert np.min(got[3]["margin"]) > 1e-9 and np.min(got[3]["gap"]) > 1e-9
    ref = brute.accept_sampled(lg, tok, par, u, 1000 + seed, T, 6)
    for a, r in zip(got[:3], ref):
        np.testing.assert_array_equal(a, r)


P4 = np.array([0.4, 0.3, 0.2, 0.1])


def _one(lg, tok, par, u, seed=0, T=1.0, Dmax=8):
    ln, path, corr = tree_accept_sampled(lg, np.array([tok]), np.array([par]),
                                         np.array([u], dtype=np.float64), seed, T, Dmax)
    return int(ln[0]), path[0][:ln[0]].tolist(), int(corr[0])


def test_thresholds_follow_the_residual():
    """Root with children of tokens 1 and 2 under p = [.4, .3, .2, .1]: the
    first child passes when u1 < p(1) = 0.3; after it is rejected the second
    is tested against the residual without token 1: u2 < 0.2 / 0.7."""
    lg = np.log(P4)[None].repeat(3, 0)[None]
    par, tok = [-1, 0, 0], [0, 1, 2]
    assert _one(lg, tok, par, [0, 0.29, 0.99])[:2] == (2, [0, 1])
    assert _one(lg, tok, par, [0, 0.31, 0.28])[:2] == (2, [0, 2])   # 0.28 * 0.7 < 0.2
    ln, path, corr = _one(lg, tok, par, [0, 0.31, 0.29])            # 0.29 * 0.7 > 0.2
    assert (ln, path) == (1, [0]) and corr in (0, 3)                # tokens 1, 2 removed
    # a repeated token is never accepted once its first occurrence failed
    par3, tok3 = [-1, 0, 0, 0], [0, 2, 2, 0]
    assert _one(lg[:, [0, 0, 0, 0]], tok3, par3, [0, 0.5, 0.0, 0.9])[:2] == (1, [0])
    assert _one(lg[:, [0, 0, 0, 0]], tok3, par3, [0, 0.5, 0.0, 0.1])[:2] == (2, [0, 3])


def test_zero_uniforms_take_the_first_child_at_every_node():
    rng = np.random.default_rng(1)
    lg, tok, par, u = _case(rng, B=1, N=14, dup=False)
    ln, path, _ = tree_accept_sampled(lg, tok, par, 0 * u, 5, 1.0, 8)
    walk = [0]
    while True:
        kids = [c for c in range(1, 14) if par[0, c] == walk[-1]]
        if not kids:
            break
        walk.append(min(kids))
    assert ln[0] == len(walk) and path[0, :ln[0]].tolist() == walk


@pytest.mark.parametrize("seed", range(4))
def test_low_temperature_is_the_greedy_rule(seed):
    """As T -> 0, p_v becomes the point mass at the argmax: a child passes
    iff its token is the target's greedy prediction at its parent, and the
    correction is that prediction at the last node -- the greedy rule
    (Sec. 2.4) whenever siblings carry distinct tokens."""
    rng = np.random.default_rng(40 + seed)
    B, N, V = 4, 24, 9
    lg, tok, par, u = _case(rng, B=B, N=N, V=V, depth=6, dup=False)
    lg = np.round(lg * 4)                           # a unique maximum per row ...
    lg[np.arange(B)[:, None], np.arange(N), rng.integers(0, V, size=(B, N))] = lg.max(-1) + 1.5
    tgt = lg.argmax(-1)
    for b in range(B):                              # ... and many matching drafts
        for i in range(1, N):
            if rng.random() < 0.7:
                sib = [c for c in range(1, N) if par[b, c] == par[b, i] and c != i]
                if all(tok[b, c] != tgt[b, par[b, i]] for c in sib):
                    tok[b, i] = tgt[b, par[b, i]]
    ln, path, corr = tree_accept_sampled(lg, tok, par, u, 3, 1e-3, N)
    gl, gp, gt = tree_accept(lg, tok, par, N)
    np.testing.assert_array_equal(ln, gl)
    np.testing.assert_array_equal(path, gp)
    np.testing.assert_array_equal(corr, gt[np.arange(B), gp[np.arange(B), gl - 1]])


def test_temperature_scales_logits():
    rng = np.random.default_rng(3)
    lg, tok, par, u = _case(rng)
    a = tree_accept_sampled(lg, tok, par, u, 4, 0.5, 6)
    b = tree_accept_sampled(2 * lg, tok, par, u, 4, 1.0, 6)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_invalid_inputs():
    rng = np.random.default_rng(4)
    lg, tok, par, u = _case(rng, B=3)
    par = par.copy()
    par[0, 3] = 5                           # parent after child
    ln, path, corr = tree_accept_sampled(lg, tok, par, u, 1, 1.0, 6)
    assert ln[0] == -1 and corr[0] == -1 and (path[0] == -1).all()
    # a chain accepted end to end needs N entries: with Dmax = 3 it cannot fit
    chain = np.arange(-1, 5)[None]
    lgc = np.zeros((1, 6, 4))
    lgc[0, :, 1] = 50.0
    ln, path, corr = tree_accept_sampled(lgc, np.ones((1, 6), int), chain, np.full((1, 6), .5),
                                         1, 1.0, 3)
    assert ln[0] == -1 and corr[0] == -1 and (path[0] == -1).all()


def test_race_sampler_frequencies():
    w = np.array([0.1, 0.0, 0.45, 0.25, 0.2])
    counts = np.zeros(5)
    for s in range(4000):
        tok = race_sample(w, 0, s)[0]
        counts[tok] += 1
    freq = counts / counts.sum()
    assert counts[1] == 0
    assert np.abs(freq - w / w.sum()).max() < 0.03


def _emitted(lg, tok, par, trials, rng, k=1):
    """Frequencies of the first k emitted tokens (accepted drafts, then the
    correction) and of the last node over `trials` runs with fresh uniforms
    and seeds."""
    N = len(par)
    firsts, ends = {}, np.zeros(N)
    us = rng.random((trials, N))
    for t in range(trials):
        ln, path, corr = _one(lg, tok, par, us[t], seed=t, Dmax=N)
        emitted = tuple([tok[x] for x in path[1:]] + [corr])[:k]
        firsts[emitted] = firsts.get(emitted, 0) + 1
        ends[path[-1]] += 1
    return {key: v / trials for key, v in firsts.items()}, ends / trials


def test_two_children_emit_the_target_distribution():
    """The rule is lossless: with deterministic children (top-W drafting),
    the first emitted token follows p at the root.  (Testing each child on
    its own against a draft distribution would emit token 1 with frequency
    about 0.86 here.)"""
    rng = np.random.default_rng(5)
    lg = np.log(P4)[None].repeat(3, 0)[None]
    freq, ends = _emitted(lg, [0, 1, 2], [-1, 0, 0], 20000, rng)
    got = np.array([freq.get((y,), 0.0) for y in range(4)])
    assert np.abs(got - P4).max() < 0.012
    # closed form of the last node: child k ends the walk with p(y_k)
    np.testing.assert_allclose(ends, [0.5, 0.3, 0.2], atol=0.012)


def test_three_children_with_a_repeat_emit_the_target_distribution():
    rng = np.random.default_rng(6)
    lg = np.log(P4)[None].repeat(4, 0)[None]
    freq, ends = _emitted(lg, [0, 2, 2, 0], [-1, 0, 0, 0], 20000, rng)
    got = np.array([freq.get((y,), 0.0) for y in range(4)])
    assert np.abs(got - P4).max() < 0.012
    assert ends[2] == 0.0                        # the repeat is never accepted


def test_two_levels_follow_the_target_sequence_distribution():
    """Two emitted tokens of a depth-2 tree: P(y1, y2) = p_root(y1) p_y1(y2)
    when the tree holds node y1, and the end-node probabilities are the
    closed form prod(p on the root path) x (1 - sum of p over the distinct
    child tokens)."""
    rng = np.random.default_rng(7)
    V = 4
    par = [-1, 0, 0, 1, 1, 2]
    tok = [0, 1, 3, 0, 2, 2]
    lg = rng.normal(size=(1, 6, V))
    p = np.exp(lg[0]) / np.exp(lg[0]).sum(-1, keepdims=True)
    freq, ends = _emitted(lg, tok, par, 30000, rng, k=2)
    # joint of the first two tokens through node 1 (token 1)
    for y2 in range(V):
        assert abs(freq.get((1, y2), 0.0) - p[0, 1] * p[1, y2]) < 0.01
    # single-token outcomes are the correction at the root
    for y in (0, 2):
        assert abs(freq.get((y,), 0.0) - p[0, y]) < 0.01
    closed = np.zeros(6)
    for v in range(6):
        kids = {tok[c] for c in range(1, 6) if par[c] == v}
        pr, x = 1.0, v
        while par[x] != -1:
            pr *= p[par[x], tok[x]]
            x = par[x]
        closed[v] = pr * (1 - sum(p[v, y] for y in kids))
    assert abs(closed.sum() - 1) < 1e-12
    np.testing.assert_allclose(ends, closed, atol=0.01)


def test_random_trees_end_where_the_closed_form_says():
    rng = np.random.default_rng(8)
    for case in range(3):
        lg, tok, par, _ = _case(rng, B=1, N=9, V=5, depth=3)
        lg, tok, par = lg, tok[0].tolist(), par[0].tolist()
        p = np.exp(lg[0]) / np.exp(lg[0]).sum(-1, keepdims=True)
        closed = np.zeros(9)
        for v in range(9):
            seen, first = set(), {}
            for c in range(1, 9):
                if par[c] == v and tok[c] not in seen:
                    seen.add(tok[c])
                    first[c] = True
            pr, x, ok = 1.0, v, True
            while par[x] != -1:
                sib_first = all(tok[c] != tok[x] for c in range(1, x) if par[c] == par[x])
                ok = ok and sib_first
                pr *= p[par[x], tok[x]]
                x = par[x]
            closed[v] = (pr if ok else 0.0) * (1 - sum(p[v, y] for y in seen))
        _, ends = _emitted(lg, tok, par, 12000, rng)
        np.testing.assert_allclose(ends, closed, atol=0.015)
