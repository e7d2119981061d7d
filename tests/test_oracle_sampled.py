"""Pins of the non-greedy tree-acceptance oracle (Sec. 2.4 speculative
sampling rule along tree branches, with correction sampling) and of its
counter-based generator."""
import os

import numpy as np
import pytest

from oracle import brute
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


def _case(rng, B=3, N=10, V=6, Nd=4):
    par = np.zeros((B, N), dtype=int)
    for b in range(B):
        par[b, 0] = -1
        dep = [0]
        for i in range(1, N):
            cand = [j for j in range(i) if dep[j] < Nd]
            par[b, i] = rng.choice(cand)
            dep.append(dep[par[b, i]] + 1)
    lg = rng.normal(size=(B, N, V)) * 1.5
    dl = rng.normal(size=(B, Nd, V)) * 1.5
    tok = rng.integers(0, V, size=(B, N))
    u = rng.random((B, N))
    return lg, dl, tok, par, u


@pytest.mark.parametrize("seed", range(8))
def test_matches_path_enumeration(seed):
    rng = np.random.default_rng(seed)
    lg, dl, tok, par, u = _case(rng)
    T = [1.0, 0.7, 1.6][seed % 3]
    got = tree_accept_sampled(lg, dl, tok, par, u, 1000 + seed, T, 6, detail=True)
    assert np.min(got[3]["margin"]) > 1e-9 and np.min(got[3]["gap"]) > 1e-9
    ref = brute.accept_sampled(lg, dl, tok, par, u, 1000 + seed, T, 6)
    for a, r in zip(got[:3], ref):
        np.testing.assert_array_equal(a, r)


def test_zero_uniforms_accept_every_node():
    rng = np.random.default_rng(1)
    lg, dl, tok, par, u = _case(rng, B=1, N=12)
    ln, path, _ = tree_accept_sampled(lg, dl, tok, par, 0 * u, 5, 1.0, 8)
    depth = np.zeros(12, dtype=int)
    for i in range(1, 12):
        depth[i] = depth[par[0, i]] + 1
    deepest = int(np.argmax(depth))       # first index of the maximum depth
    assert ln[0] == depth[deepest] + 1 and path[0, ln[0] - 1] == deepest


def test_draft_equal_to_target_accepts_a_chain():
    """q of depth d equal to p at the depth-(d-1) node: every ratio is 1."""
    rng = np.random.default_rng(2)
    N, V = 6, 9
    par = np.arange(-1, N - 1)[None]
    lg = rng.normal(size=(1, N, V))
    dl = lg[:, :N - 1].copy()
    tok = rng.integers(0, V, size=(1, N))
    u = np.full((1, N), 0.999999)
    ln, path, corr = tree_accept_sampled(lg, dl, tok, par, u, 9, 1.0, N)
    assert ln[0] == N and path[0].tolist() == list(range(N))
    # the last node is a leaf: its correction comes from p there
    tok_ref = race_sample(np.exp(lg[0, N - 1]) / np.exp(lg[0, N - 1]).sum(), 0, 9)[0]
    assert corr[0] == tok_ref


def test_temperature_scales_logits():
    rng = np.random.default_rng(3)
    lg, dl, tok, par, u = _case(rng)
    a = tree_accept_sampled(lg, dl, tok, par, u, 4, 0.5, 6)
    b = tree_accept_sampled(2 * lg, 2 * dl, tok, par, u, 4, 1.0, 6)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_invalid_inputs():
    rng = np.random.default_rng(4)
    lg, dl, tok, par, u = _case(rng, B=3)
    par = par.copy()
    par[0, 3] = 5                           # parent after child
    ln, path, corr = tree_accept_sampled(lg, dl[:, :2], tok, par, u, 1, 1.0, 6)
    assert ln[0] == -1 and corr[0] == -1 and (path[0] == -1).all()
    # dl has 2 depths but the trees reach depth 4: too deep for the draft
    assert (ln == -1).all() and (corr == -1).all()


def test_race_sampler_frequencies():
    w = np.array([0.1, 0.0, 0.45, 0.25, 0.2])
    counts = np.zeros(5)
    for s in range(4000):
        tok = race_sample(w, 0, s)[0]
        counts[tok] += 1
    freq = counts / counts.sum()
    assert counts[1] == 0
    assert np.abs(freq - w / w.sum()).max() < 0.03


def test_emitted_token_follows_the_target():
    """Speculative sampling keeps the target distribution: with one draft
    node whose token is drawn from q, the first emitted token (the draft if
    accepted, else the correction) is distributed as p at the root."""
    V = 5
    rng = np.random.default_rng(5)
    lg = rng.normal(size=(1, 2, V))
    dl = rng.normal(size=(1, 1, V))
    p = np.exp(lg[0, 0]) / np.exp(lg[0, 0]).sum()
    q = np.exp(dl[0, 0]) / np.exp(dl[0, 0]).sum()
    par = np.array([[-1, 0]])
    counts = np.zeros(V)
    trials = 20000
    ys = rng.choice(V, size=trials, p=q)
    us = rng.random(trials)
    for t in range(trials):
        tok = np.array([[0, ys[t]]])
        ln, path, corr = tree_accept_sampled(lg, dl, tok, par, np.array([[0.0, us[t]]]), t,
                                             1.0, 2)
        counts[ys[t] if ln[0] == 2 else corr[0]] += 1
    assert np.abs(counts / trials - p).max() < 0.015
