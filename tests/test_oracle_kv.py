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
