"""Pins of the cache-commit oracle (App. E: the accepted path is committed to
the cache; paged caches): element-wise brute force, the paged form against
the contiguous form through an independent gather, and the readings for
failed or overflowing commits."""
import numpy as np
import pytest

from oracle import kv_commit


def _case(rng, B=3, N=9, Hkv=2, D=4, Lmax=24):
    kc = rng.normal(size=(B, Lmax, Hkv, D))
    vc = rng.normal(size=(B, Lmax, Hkv, D))
    kt = rng.normal(size=(B, N, Hkv, D))
    vt = rng.normal(size=(B, N, Hkv, D))
    return kc, vc, kt, vt


def test_commit_matches_elementwise_loops():
    rng = np.random.default_rng(0)
    kc, vc, kt, vt = _case(rng)
    B, Lmax, Hkv, D = kc.shape
    path = np.array([[0, 3, 5, -1], [0, 1, -1, -1], [0, 2, 4, 8]])
    accept_len = np.array([3, 2, 4])
    kv_len = np.array([5, 0, 20])
    nk, nv, nl = kv_commit.commit_path(kc, vc, kt, vt, path, accept_len, kv_len)
    for b in range(B):
        for t in range(Lmax):
            for h in range(Hkv):
                for d in range(D):
                    j = t - kv_len[b]
                    if 0 <= j < accept_len[b]:
                        ek, ev = kt[b, path[b][j], h, d], vt[b, path[b][j], h, d]
                    else:
                        ek, ev = kc[b, t, h, d], vc[b, t, h, d]
                    assert nk[b, t, h, d] == ek and nv[b, t, h, d] == ev
    assert nl.tolist() == [8, 2, 24]


def test_failed_or_overflowing_commit_leaves_the_sequence():
    rng = np.random.default_rng(1)
    kc, vc, kt, vt = _case(rng)
    path = np.array([[0, 1, -1], [-1, -1, -1], [0, 4, 6]])
    accept_len = np.array([2, -1, 3])
    kv_len = np.array([23, 7, 10])        # sequence 0 would pass Lmax = 24
    nk, nv, nl = kv_commit.commit_path(kc, vc, kt, vt, path, accept_len, kv_len)
    assert nl.tolist() == [23, 7, 13]
    np.testing.assert_array_equal(nk[:2], kc[:2])
    np.testing.assert_array_equal(nv[:2], vc[:2])
    np.testing.assert_array_equal(nk[2, 10:13], kt[2, [0, 4, 6]])


@pytest.mark.parametrize("bs", [1, 4, 8])
def test_paged_commit_matches_contiguous(bs):
    rng = np.random.default_rng(bs)
    B, N, Hkv, D, nblk = 3, 7, 2, 3, 6
    cap = nblk * bs
    kt = rng.normal(size=(B, N, Hkv, D))
    vt = rng.normal(size=(B, N, Hkv, D))
    num = B * nblk + 5
    kp = rng.normal(size=(num, bs, Hkv, D))
    vp = rng.normal(size=(num, bs, Hkv, D))
    bt = rng.permutation(num)[:B * nblk].reshape(B, nblk)   # blocks of a sequence anywhere
    kv_len = rng.integers(0, cap - 2, size=B)
    accept_len = np.array([1, 3, 2])
    path = np.array([[0, -1, -1], [0, 2, 5], [0, 6, -1]])
    pk, pv, pl = kv_commit.commit_path_paged(kp, vp, bt, kt, vt, path, accept_len, kv_len, cap)
    ck, cv, cl = kv_commit.commit_path(kv_commit.gather_paged(kp, bt, nblk),
                                       kv_commit.gather_paged(vp, bt, nblk), kt, vt, path,
                                       accept_len, kv_len)
    np.testing.assert_array_equal(kv_commit.gather_paged(pk, bt, nblk), ck)
    np.testing.assert_array_equal(kv_commit.gather_paged(pv, bt, nblk), cv)
    np.testing.assert_array_equal(pl, cl)
    # pool blocks no sequence uses are untouched
    unused = np.setdiff1d(np.arange(num), bt.ravel())
    np.testing.assert_array_equal(pk[unused], kp[unused])


def test_gather_paged_elementwise():
    rng = np.random.default_rng(5)
    pool = rng.normal(size=(10, 4, 1, 2))
    bt = np.array([[3, 9, 0], [7, 1, 2]])
    g = kv_commit.gather_paged(pool, bt, 3)
    for b in range(2):
        for t in range(12):
            np.testing.assert_array_equal(g[b, t], pool[bt[b, t // 4], t % 4])


def _tree_paths(rng, B, N):
    """Random trees (parent before child) and one root-to-node path each,
    root first, padded with -1 to N entries."""
    from paper_2606_18394_amd import synth
    par = np.stack([synth.random_tree(rng, N, depth=min(N - 1, 6), branching=3)
                    for _ in range(B)])
    path = np.full((B, N), -1)
    n = np.zeros(B, dtype=np.int64)
    for b in range(B):
        u, p = int(rng.integers(0, N)), []
        while u != -1:
            p.append(u)
            u = int(par[b, u])
        p.reverse()
        path[b, :len(p)] = p
        n[b] = len(p)
    return par, path, n


def test_tree_tail_is_the_slice_after_the_context():
    rng = np.random.default_rng(11)
    c = rng.normal(size=(2, 20, 1, 3))
    t = kv_commit.tree_tail(c, np.array([4, 11]), 6)
    for b, kl in enumerate([4, 11]):
        for i in range(6):
            np.testing.assert_array_equal(t[b, i], c[b, kl + i])


@pytest.mark.parametrize("seed", range(6))
def test_tail_commit_matches_in_place_moves(seed):
    from oracle import brute
    rng = np.random.default_rng(100 + seed)
    B, N, Lmax = 4, 12, 40
    _, path, n = _tree_paths(rng, B, N)
    kc = rng.normal(size=(B, Lmax, 2, 3))
    vc = rng.normal(size=(B, Lmax, 2, 3))
    kl = rng.integers(0, Lmax - N + 1, size=B)
    nk, nv, nl = kv_commit.commit_path_tail(kc, vc, path, n, kl, N)
    np.testing.assert_array_equal(nk, brute.commit_tail_in_place(kc, path, n, kl))
    np.testing.assert_array_equal(nv, brute.commit_tail_in_place(vc, path, n, kl))
    np.testing.assert_array_equal(nl, kl + n)


def test_tail_commit_reads_rows_before_overwriting_them():
    """path [0, 2, 5]: row kl+1 takes row kl+2, which row kl+2 then takes
    from row kl+5; a commit that wrote before reading would copy the wrong
    row into kl+1."""
    c = np.arange(10, dtype=float).reshape(1, 10, 1, 1)
    nk, _, nl = kv_commit.commit_path_tail(c, c, np.array([[0, 2, 5]]), np.array([3]),
                                           np.array([2]), 6)
    assert nk[0, :, 0, 0].tolist() == [0, 1, 2, 4, 7, 5, 6, 7, 8, 9]
    assert nl.tolist() == [5]


def test_tail_commit_without_room_leaves_the_sequence():
    rng = np.random.default_rng(3)
    c = rng.normal(size=(2, 10, 1, 2))
    path = np.array([[0, 1, -1], [0, 1, 2]])
    nk, _, nl = kv_commit.commit_path_tail(c, c, path, np.array([2, 3]), np.array([5, 4]), 6)
    np.testing.assert_array_equal(nk[0], c[0])      # 5 + 6 > 10: no room for the tree
    assert nl.tolist() == [5, 7]
    np.testing.assert_array_equal(nk[1, 4:7], c[1, [4, 5, 6]])
