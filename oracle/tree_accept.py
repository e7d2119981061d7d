"""Oracle of greedy tree acceptance (test infrastructure only).

What it computes (Sec. 2.4 greedy rule; App. E): the target's greedy
prediction at every node is the argmax of that node's logits; a draft node is
accepted when its token equals the prediction at its parent and its parent is
accepted (the root, the already-sampled token, is always accepted); the
result is the deepest fully accepted root-to-node path.  The prediction at the
path's last node is the correction token.

Readings where the paper is silent:
  * argmax ties go to the lowest vocabulary index, values compared as numbers
    (-0.0 equals +0.0);
  * among equally deep accepted nodes the lowest node index wins;
  * accept_len counts path entries including the root;
  * path is root first, padded with -1 to Dmax entries;
  * an invalid tree (parent[0] != -1 or parent[i] outside [0, i)) or a path
    longer than Dmax gives accept_len = -1 and path all -1; the argmax output
    is still produced.
"""
from __future__ import annotations

import numpy as np

from .tree_attention import tree_structure


def target_argmax(logits) -> np.ndarray:
    """First index of the maximum of each row: [B,N,V] -> [B,N] int32."""
    lg = np.asarray(logits, dtype=np.float64)
    return np.argmax(lg, axis=-1).astype(np.int32)


def tree_accept(logits, draft_tok, parent, Dmax: int):
    """Returns (accept_len [B] int32, path [B,Dmax] int32, tgt [B,N] int32)."""
    tgt = target_argmax(logits)
    draft_tok = np.asarray(draft_tok)
    parent = np.asarray(parent)
    B, N = parent.shape
    if Dmax < 1:
        raise ValueError("Dmax must be >= 1")
    accept_len = np.full(B, -1, dtype=np.int32)
    path = np.full((B, Dmax), -1, dtype=np.int32)
    for b in range(B):
        valid, _, depth = tree_structure(parent[b])
        if not valid:
            continue
        acc = np.zeros(N, dtype=bool)
        acc[0] = True
        for i in range(1, N):
            p = parent[b, i]
            acc[i] = acc[p] and draft_tok[b, i] == tgt[b, p]
        best = 0
        for i in range(1, N):
            if acc[i] and depth[i] > depth[best]:
                best = i
        length = int(depth[best]) + 1
        if length > Dmax:
            continue
        walk = [best]
        while walk[-1] != 0:
            walk.append(int(parent[b, walk[-1]]))
        walk.reverse()
        accept_len[b] = length
        path[b, :length] = walk
    return accept_len, path, tgt
