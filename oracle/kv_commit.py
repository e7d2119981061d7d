"""Oracle of the cache side of a verification step (test infrastructure only).

What it computes (App. E, "vLLM Implementation Details": the accepted path is
committed to the cache, and the verification kernel reads a paged cache):

  commit_path   the K and V of the accepted path's nodes (root first) are
                appended to the sequence's cache at positions kv_len ..
                kv_len + accept_len - 1, and kv_len grows by accept_len.
  gather_paged  the contiguous cache that a paged cache (a pool of fixed-size
                blocks and a per-sequence block table) stands for.
  tree_tail,    the tree-tail layout, in which the draft nodes' K/V were
  commit_path_tail  written to the cache right after the context (node i at
                position kv_len + i) before verification: the tree K/V are
                that slice, and committing moves the accepted path's rows
                down to kv_len .. kv_len + accept_len - 1.

Readings where the paper is silent:
  * the root (the token sampled by the previous step) is committed with the
    accepted drafts: its K/V are computed by this verification pass;
  * a sequence whose acceptance failed (accept_len < 1) or whose commit would
    pass the cache capacity is left unchanged (cache and kv_len);
  * paged caches use blocks of block_size consecutive positions; logical
    block j of sequence b is pool block block_table[b, j];
  * in the tree-tail layout a sequence needs kv_len + N <= capacity; a
    sequence with less room is left unchanged by the commit.
"""
from __future__ import annotations

import numpy as np


def commit_path(k_cache, v_cache, k_tree, v_tree, path, accept_len, kv_len):
    """Contiguous caches [B, Lmax, Hkv, D]; tree K/V [B, N, Hkv, D];
    path [B, Dmax]; accept_len [B]; kv_len [B].  Returns new copies
    (k_cache, v_cache, kv_len)."""
    kc, vc = np.array(k_cache, copy=True), np.array(v_cache, copy=True)
    kl = np.array(kv_len, dtype=np.int64, copy=True)
    B, Lmax = kc.shape[0], kc.shape[1]
    for b in range(B):
        n = int(accept_len[b])
        if n < 1 or kl[b] + n > Lmax:
            continue
        for j in range(n):
            node = int(path[b][j])
            kc[b, kl[b] + j] = k_tree[b, node]
            vc[b, kl[b] + j] = v_tree[b, node]
        kl[b] += n
    return kc, vc, kl


def gather_paged(pool, block_table, n_blocks):
    """pool [num_blocks, block_size, Hkv, D], block_table [B, max_blocks]:
    the first n_blocks blocks of every sequence as a contiguous
    [B, n_blocks * block_size, Hkv, D] array."""
    pool = np.asarray(pool)
    bt = np.asarray(block_table)
    B = bt.shape[0]
    bs = pool.shape[1]
    out = np.empty((B, n_blocks * bs) + pool.shape[2:], dtype=pool.dtype)
    for b in range(B):
        for j in range(n_blocks):
            out[b, j * bs:(j + 1) * bs] = pool[bt[b, j]]
    return out


def commit_path_paged(k_pool, v_pool, block_table, k_tree, v_tree, path, accept_len, kv_len,
                      capacity):
    """Paged form of commit_path: position t of sequence b lives at
    pool[block_table[b, t // bs], t % bs].  capacity = positions a sequence
    may hold.  Returns new copies (k_pool, v_pool, kv_len)."""
    kp, vp = np.array(k_pool, copy=True), np.array(v_pool, copy=True)
    kl = np.array(kv_len, dtype=np.int64, copy=True)
    bt = np.asarray(block_table)
    bs = kp.shape[1]
    for b in range(bt.shape[0]):
        n = int(accept_len[b])
        if n < 1 or kl[b] + n > capacity:
            continue
        for j in range(n):
            t = int(kl[b]) + j
            node = int(path[b][j])
            kp[bt[b, t // bs], t % bs] = k_tree[b, node]
            vp[bt[b, t // bs], t % bs] = v_tree[b, node]
        kl[b] += n
    return kp, vp, kl


def tree_tail(cache, kv_len, n_nodes):
    """Tree-tail layout: the [B, N, ...] tree K (or V) a contiguous cache holds
    at positions kv_len[b] .. kv_len[b] + N - 1."""
    cache = np.asarray(cache)
    out = np.empty((cache.shape[0], n_nodes) + cache.shape[2:], dtype=cache.dtype)
    for b in range(cache.shape[0]):
        kl = int(kv_len[b])
        out[b] = cache[b, kl:kl + n_nodes]
    return out


def commit_path_tail(k_cache, v_cache, path, accept_len, kv_len, n_nodes):
    """commit_path in the tree-tail layout: the tree K/V are the cache rows
    kv_len .. kv_len + N - 1 as they are before the commit.  Returns new
    copies (k_cache, v_cache, kv_len)."""
    Lmax = np.asarray(k_cache).shape[1]
    kl = np.asarray(kv_len, dtype=np.int64)
    room = kl + n_nodes <= Lmax
    safe_kl = np.where(room, kl, 0)                 # only read where there is room
    kt = tree_tail(k_cache, safe_kl, n_nodes)
    vt = tree_tail(v_cache, safe_kl, n_nodes)
    n = np.where(room, np.asarray(accept_len), 0)   # no room: left unchanged
    return commit_path(k_cache, v_cache, kt, vt, path, n, kv_len)
