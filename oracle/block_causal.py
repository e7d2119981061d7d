"""fp64 oracle of attention under the draft head's training mask (test
infrastructure only).

What it computes (App. "Training Details" and its training-mask figure): a
training example samples A anchor positions in its sequence.  Each anchor
starts a block of S positions: position 0 is the anchor token, the others are
mask tokens whose future tokens the head predicts.  A query at position j of
block k attends to

  * the verified prefix: context rows t < anchors[k] (the context K/V are
    the target-model features of the sequence), and
  * positions 0 .. j of its own block (the anchor and earlier positions),

and to nothing else: no later position, no other block.  Scores are
Q K^T / sqrt(d) with d the head dimension, then softmax and the weighted sum
of V, exactly as in the tree-verification attention.

Readings where the paper is silent:
  * "the prefix" of a block is the context strictly before its anchor; the
    anchor itself is block position 0, so it is seen once;
  * anchors are clamped into [0, L];
  * grouped-query attention maps query head h to KV head floor(h / G).

The full [A*S, L + A*S] mask is materialised from the rule above; nothing is
blocked, fused or reordered.
"""
from __future__ import annotations

import numpy as np


def training_mask(anchors, L: int, S: int) -> np.ndarray:
    """Visibility [A*S, L + A*S]: row k*S + j is position j of block k;
    column t < L is context row t, column L + k*S + i is position i of
    block k."""
    A = len(anchors)
    m = np.zeros((A * S, L + A * S), dtype=bool)
    for k in range(A):
        a = min(max(int(anchors[k]), 0), L)
        for j in range(S):
            r = k * S + j
            m[r, :a] = True
            m[r, L + k * S:L + k * S + j + 1] = True
    return m


def block_causal_attention(q, k_ctx, v_ctx, k_blk, v_blk, anchors, scale=None):
    """q [B, A, S, Hq, D]; k_ctx, v_ctx [B, L, Hkv, D]; k_blk, v_blk
    [B, A, S, Hkv, D]; anchors [B, A].  float64 arrays.  Returns
    [B, A, S, Hq, D]."""
    q = np.asarray(q, dtype=np.float64)
    B, A, S, Hq, D = q.shape
    L, Hkv = k_ctx.shape[1], k_ctx.shape[2]
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    out = np.zeros_like(q)
    for b in range(B):
        m = training_mask(anchors[b], L, S)
        kb = np.asarray(k_blk[b], dtype=np.float64).reshape(A * S, Hkv, D)
        vb = np.asarray(v_blk[b], dtype=np.float64).reshape(A * S, Hkv, D)
        keys = np.concatenate([np.asarray(k_ctx[b], dtype=np.float64), kb], axis=0)
        vals = np.concatenate([np.asarray(v_ctx[b], dtype=np.float64), vb], axis=0)
        qb = q[b].reshape(A * S, Hq, D)
        for h in range(Hq):
            g = h // G
            s = (qb[:, h, :] @ keys[:, g, :].T) * scale
            s = np.where(m, s, -np.inf)
            s = s - s.max(axis=1, keepdims=True)
            w = np.exp(s)
            w /= w.sum(axis=1, keepdims=True)
            out[b, :, :, h, :] = (w @ vals[:, g, :]).reshape(A, S, D)
    return out
