"""Checks of the seeded input generator (shapes, tree caps, determinism)."""
import numpy as np
import pytest

import oracle
from paper_2606_18394_amd import synth


def _depths(parent):
    d = np.zeros(len(parent), dtype=int)
    for i in range(1, len(parent)):
        d[i] = d[parent[i]] + 1
    return d


def test_bf16_rne():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1000.0, 1.0 + 2 ** -9],
                 dtype=np.float32)
    got = synth.bf16_bits(x)
    # 1+2^-8 is a tie -> even (1.0); 1+3*2^-8 is a tie -> even (1+2^-6... 1.015625)
    assert got.tolist() == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x447A, 0x3F80]
    import torch
    y = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    ref = torch.from_numpy(y).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(synth.bf16_bits(y), ref)


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workload_trees(name):
    w = synth.WORKLOADS[name]
    rng = np.random.Generator(np.random.PCG64(w.seed))
    for _ in range(3):
        p = synth.random_tree(rng, w.N, w.depth, w.branching, w.spine)
        assert p[0] == -1 and all(0 <= p[i] < i for i in range(1, w.N))
        d = _depths(p)
        assert d.max() <= w.depth
        if w.spine:
            assert d.max() == w.depth
        if w.branching is not None:
            assert np.bincount(p[1:], minlength=w.N).max() <= w.branching


def test_draw_small_and_deterministic():
    w = synth.WORKLOADS["tiny"]
    a, b = synth.draw(w), synth.draw(w)
    for k in ["parent", "kv_len", "q", "k_cache", "logits", "match", "rand_tok"]:
        np.testing.assert_array_equal(a[k], b[k])
    assert a["q"].shape == (1, 16, 4, 64) and a["q"].dtype == np.uint16
    assert a["k_cache"].shape == (1, 256, 2, 64)
    assert a["logits"].dtype == np.float32 and a["logits"].shape == (1, 16, 1024)
    c = synth.draw(w, seed=5)
    assert not np.array_equal(a["q"], c["q"])


def test_ragged_kv_len_and_poison():
    w = synth.with_shape(synth.WORKLOADS["batched_30b_a3b"], L=64, ragged=(3, 64),
                         V=16, D=16)
    x = synth.draw(w)
    assert x["kv_len"].min() >= 3 and x["kv_len"].max() <= 64
    for b in range(w.B):
        assert (x["k_cache"][b, x["kv_len"][b]:] == synth.POISON_BF16).all()
        assert (x["v_cache"][b, x["kv_len"][b]:] == synth.POISON_BF16).all()


def test_match_rate():
    w = synth.with_shape(synth.WORKLOADS["qwen3_8b"], V=64, L=16, N=64, B=1)
    rng = np.random.default_rng(1)
    B, N, V, p = 64, 64, 64, 0.6
    trees = np.stack([synth.random_tree(rng, N, 8, 4, True) for _ in range(B)])
    logits = rng.standard_normal((B, N, V))
    tgt = oracle.target_argmax(logits)
    draft = synth.draft_tokens(trees, tgt, rng.random((B, N)) < p, rng.integers(0, V, (B, N)))
    hit = np.mean([draft[b, i] == tgt[b, trees[b, i]] for b in range(B) for i in range(1, N)])
    assert abs(hit - (p + (1 - p) / V)) < 0.03
