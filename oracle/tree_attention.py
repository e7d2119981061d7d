"""fp64 oracle of tree-verification attention (test infrastructure only).

What it computes (Sec. 2.2, the tree-causal mask and the masked attention
equations): for draft-tree node v, its query attends to every prefix (KV
cache) position and to the tree nodes u in Anc(v) plus v itself; every other
tree node is masked with -inf.  The score is Q_v K^T / sqrt(d) with d the head
dimension, followed by a softmax and a weighted sum of V.

Readings where the paper is silent:
  * grouped-query attention maps query head h to KV head floor(h / G),
    G = Hq / Hkv (contiguous groups);
  * the cache is padded to Lmax and positions >= kv_len[b] are invisible;
  * parent[0] = -1 and 0 <= parent[i] < i (children follow their parent as in
    Alg. 1); any other tree makes every output row of that sequence NaN.

The full [N, Lmax + N] mask is materialised explicitly; nothing is blocked,
fused or reordered.
"""
from __future__ import annotations

import numpy as np


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64, exactly."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def tree_structure(parent_row: np.ndarray):
    """Validate one sequence's parent array; return (valid, anc, depth).

    anc[i, u] is True iff u is node i or one of its ancestors.  Built by
    the recursion anc[i] = anc[parent[i]] with bit i added, in node order,
    which is well defined because parents precede children.
    """
    p = np.asarray(parent_row, dtype=np.int64)
    n = p.shape[0]
    anc = np.zeros((n, n), dtype=bool)
    depth = np.zeros(n, dtype=np.int64)
    if n == 0 or p[0] != -1:
        return False, anc, depth
    anc[0, 0] = True
    for i in range(1, n):
        if not (0 <= p[i] < i):
            return False, anc, depth
        anc[i] = anc[p[i]]
        anc[i, i] = True
        depth[i] = depth[p[i]] + 1
    return True, anc, depth


def full_mask(parent_row: np.ndarray, kv_len: int, Lmax: int) -> np.ndarray:
    """Visibility of every key for every node: [N, Lmax + N] bool.

    Column j < Lmax is cache position j (visible iff j < kv_len, the prefix
    being visible to all nodes); column Lmax + u is tree node u.
    """
    valid, anc, _ = tree_structure(parent_row)
    n = len(parent_row)
    m = np.zeros((n, Lmax + n), dtype=bool)
    m[:, :kv_len] = True
    m[:, Lmax:] = anc
    return m


def tree_attention(q, k_cache, v_cache, k_tree, v_tree, parent, kv_len=None,
                   scale=None, nodes=None, heads=None) -> np.ndarray:
    """Tree attention output in fp64.

    Shapes: q [B,N,Hq,D]; k_cache, v_cache [B,Lmax,Hkv,D]; k_tree, v_tree
    [B,N,Hkv,D]; parent [B,N]; kv_len [B] or None (= Lmax).  Arrays may be
    any float type; they are upcast exactly to fp64.  ``nodes``/``heads``
    restrict the output to a subset of rows (the result is the same as
    slicing the full output).  Returns [B, len(nodes), len(heads), D].
    """
    q = np.asarray(q, dtype=np.float64)
    k_cache = np.asarray(k_cache, dtype=np.float64)
    v_cache = np.asarray(v_cache, dtype=np.float64)
    k_tree = np.asarray(k_tree, dtype=np.float64)
    v_tree = np.asarray(v_tree, dtype=np.float64)
    parent = np.asarray(parent)
    B, N, Hq, D = q.shape
    Lmax, Hkv = k_cache.shape[1], k_cache.shape[2]
    if Hq % Hkv != 0:
        raise ValueError("Hq must be a multiple of Hkv")
    if k_cache.shape != (B, Lmax, Hkv, D) or v_cache.shape != k_cache.shape:
        raise ValueError("cache shape mismatch")
    if k_tree.shape != (B, N, Hkv, D) or v_tree.shape != k_tree.shape:
        raise ValueError("tree K/V shape mismatch")
    if parent.shape != (B, N):
        raise ValueError("parent shape mismatch")
    G = Hq // Hkv
    if kv_len is None:
        kv_len = np.full(B, Lmax, dtype=np.int64)
    kv_len = np.asarray(kv_len, dtype=np.int64)
    if np.any(kv_len < 0) or np.any(kv_len > Lmax):
        raise ValueError("kv_len out of range")
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    nodes = np.arange(N) if nodes is None else np.asarray(nodes)
    heads = np.arange(Hq) if heads is None else np.asarray(heads)

    out = np.empty((B, len(nodes), len(heads), D), dtype=np.float64)
    for b in range(B):
        valid, _, _ = tree_structure(parent[b])
        if not valid:
            out[b] = np.nan
            continue
        mask = full_mask(parent[b], int(kv_len[b]), Lmax)[nodes]   # [n, Lmax+N]
        for hi, h in enumerate(heads):
            g = h // G
            kf = np.concatenate([k_cache[b, :, g, :], k_tree[b, :, g, :]], axis=0)
            vf = np.concatenate([v_cache[b, :, g, :], v_tree[b, :, g, :]], axis=0)
            s = (q[b, nodes, h, :] @ kf.T) * scale
            s = np.where(mask, s, -np.inf)
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p = p / p.sum(axis=1, keepdims=True)
            out[b, :, hi, :] = p @ vf
    return out
