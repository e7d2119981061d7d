"""Pins of the training-mask attention oracle (App. Training Details: each
block sees the prefix before its anchor and its own anchor and earlier
positions, never another block): brute force, library special cases, a
closed form and invariances."""
import numpy as np
import pytest
import torch

from oracle import block_causal, brute
from oracle.tree_attention import tree_attention


def _inputs(rng, B=2, A=3, S=4, Hq=4, Hkv=2, D=8, L=10):
    q = rng.normal(size=(B, A, S, Hq, D))
    kc = rng.normal(size=(B, L, Hkv, D))
    vc = rng.normal(size=(B, L, Hkv, D))
    kb = rng.normal(size=(B, A, S, Hkv, D))
    vb = rng.normal(size=(B, A, S, Hkv, D))
    return q, kc, vc, kb, vb


def test_mask_of_a_small_example():
    # L = 4 context rows, blocks of S = 2, anchors at 1 and 3
    m = block_causal.training_mask([1, 3], 4, 2)
    expect = np.array([
        # ctx0 ctx1 ctx2 ctx3 | b0p0 b0p1 | b1p0 b1p1
        [1, 0, 0, 0, 1, 0, 0, 0],
        [1, 0, 0, 0, 1, 1, 0, 0],
        [1, 1, 1, 0, 0, 0, 1, 0],
        [1, 1, 1, 0, 0, 0, 1, 1],
    ], dtype=bool)
    np.testing.assert_array_equal(m, expect)


def test_matches_brute_force():
    rng = np.random.default_rng(0)
    q, kc, vc, kb, vb = _inputs(rng)
    anchors = np.array([[0, 10, 4], [-3, 15, 7]])   # clamped into [0, L]
    got = block_causal.block_causal_attention(q, kc, vc, kb, vb, anchors)
    ref = brute.block_causal(q, kc, vc, kb, vb, anchors)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_single_block_at_zero_is_causal_self_attention():
    rng = np.random.default_rng(1)
    q, kc, vc, kb, vb = _inputs(rng, B=1, A=1, S=7, Hq=2, Hkv=2, D=16, L=5)
    got = block_causal.block_causal_attention(q, kc, vc, kb, vb, np.array([[0]]))
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x[0, 0].transpose(1, 0, 2)))
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(kb), t(vb), is_causal=True)
    np.testing.assert_allclose(got[0, 0], ref.numpy().transpose(1, 0, 2), rtol=1e-12, atol=1e-12)


def test_blocks_of_one_are_decode_over_prefix_and_anchor():
    rng = np.random.default_rng(2)
    q, kc, vc, kb, vb = _inputs(rng, B=1, A=4, S=1, Hq=3, Hkv=3, D=8, L=9)
    anchors = np.array([[0, 3, 9, 5]])
    got = block_causal.block_causal_attention(q, kc, vc, kb, vb, anchors)
    for k, a in enumerate(anchors[0]):
        keys = np.concatenate([kc[0, :a], kb[0, k]], axis=0).transpose(1, 0, 2)
        vals = np.concatenate([vc[0, :a], vb[0, k]], axis=0).transpose(1, 0, 2)
        qq = q[0, k].transpose(1, 0, 2)                      # [H, 1, D]
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(qq), torch.from_numpy(np.ascontiguousarray(keys)),
            torch.from_numpy(np.ascontiguousarray(vals)))
        np.testing.assert_allclose(got[0, k], ref.numpy().transpose(1, 0, 2), rtol=1e-12,
                                   atol=1e-12)


def test_zero_keys_average_the_visible_values():
    rng = np.random.default_rng(3)
    q, kc, vc, kb, vb = _inputs(rng, B=1, A=3, S=5, Hq=4, Hkv=1, D=6, L=12)
    anchors = np.array([[2, 0, 12]])
    got = block_causal.block_causal_attention(q, 0 * kc, vc, 0 * kb, vb, anchors)
    for k, a in enumerate(anchors[0]):
        for j in range(5):
            mean = (vc[0, :a, 0].sum(axis=0) + vb[0, k, :j + 1, 0].sum(axis=0)) / (a + j + 1)
            for h in range(4):
                np.testing.assert_allclose(got[0, k, j, h], mean, rtol=1e-12, atol=1e-12)


def test_blocks_and_later_context_are_invisible():
    rng = np.random.default_rng(4)
    q, kc, vc, kb, vb = _inputs(rng, B=1, A=3, S=4, L=16)
    anchors = np.array([[5, 9, 2]])
    base = block_causal.block_causal_attention(q, kc, vc, kb, vb, anchors)
    kb2, vb2 = kb.copy(), vb.copy()
    kb2[0, 1] *= 1000.0
    vb2[0, 1] += 1000.0
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[0, 9:] *= 1000.0                  # at or after every other block's anchor
    vc2[0, 9:] += 1000.0
    pert = block_causal.block_causal_attention(q, kc2, vc2, kb2, vb2, anchors)
    for k in (0, 2):                      # blocks 0 and 2 see neither change
        np.testing.assert_array_equal(pert[0, k], base[0, k])
    assert np.abs(pert[0, 1] - base[0, 1]).max() > 1.0


@pytest.mark.parametrize("seed", range(3))
def test_equals_chain_trees_over_the_prefix(seed):
    """Each block is a chain tree whose cache is the prefix before its
    anchor: the tree-verification oracle gives the same numbers."""
    rng = np.random.default_rng(10 + seed)
    B, A, S, Hq, Hkv, D, L = 2, 3, 5, 4, 2, 8, 11
    q, kc, vc, kb, vb = _inputs(rng, B, A, S, Hq, Hkv, D, L)
    anchors = rng.integers(0, L + 1, size=(B, A))
    got = block_causal.block_causal_attention(q, kc, vc, kb, vb, anchors)
    chain = np.arange(-1, S - 1)
    for b in range(B):
        for k in range(A):
            ref = tree_attention(
                q[b, k][None], kc[b][None], vc[b][None], kb[b, k][None], vb[b, k][None],
                chain[None], np.array([anchors[b, k]]))
            np.testing.assert_allclose(got[b, k], ref[0], rtol=1e-12, atol=1e-12)
