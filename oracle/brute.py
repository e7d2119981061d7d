"""Pure-Python brute force for tiny inputs (test infrastructure only).

Independent constructions used to pin the oracle:
  * attention: the visible key list of node i is built by walking parent
    pointers from i to the root (not from the ancestor matrix), scores and
    the softmax use Python floats and math.exp, no numpy;
  * acceptance: every root-to-node path is enumerated explicitly and checked
    token by token against a loop argmax; the best path is chosen by
    (length, then lowest end node);
  * top-W: Python sort on (value, index) and an exactly summed log-sum-exp;
  * tree building: the full W-ary tree is enumerated and its nodes visited in
    descending score order, with no priority queue;
  * tree-tail commit: rows moved in place one at a time, with no snapshot of
    the tree rows;
  * training-mask attention: the visible key list of each query is built
    from the block rule directly, in Python floats;
  * sampled acceptance: each node's test and its siblings' evaluated on
    their own, every root-to-node path checked for being taken end to end
    (no walk), Python-float softmaxes, the correction by a Python-loop race
    over scalar Philox words.
"""
from __future__ import annotations

import math

import numpy as np


def _valid_tree(par):
    if len(par) == 0 or par[0] != -1:
        return False
    return all(0 <= par[i] < i for i in range(1, len(par)))


def _root_path(par, i):
    """Nodes from the root to i (inclusive), by walking parents."""
    out = [i]
    while par[out[-1]] != -1:
        out.append(par[out[-1]])
    return out[::-1]


def attention(q, k_cache, v_cache, k_tree, v_tree, parent, kv_len, scale=None):
    """Nested-list (or array) inputs; returns nested lists [B][N][Hq][D]."""
    B, N, Hq, D = len(q), len(q[0]), len(q[0][0]), len(q[0][0][0])
    Hkv = len(k_cache[0][0])
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    out = []
    for b in range(B):
        par = [int(x) for x in parent[b]]
        ok = _valid_tree(par)
        ob = []
        for i in range(N):
            oi = []
            for h in range(Hq):
                if not ok:
                    oi.append([float("nan")] * D)
                    continue
                g = h // G
                keys, vals = [], []
                for j in range(int(kv_len[b])):
                    keys.append([float(x) for x in k_cache[b][j][g]])
                    vals.append([float(x) for x in v_cache[b][j][g]])
                for u in _root_path(par, i):
                    keys.append([float(x) for x in k_tree[b][u][g]])
                    vals.append([float(x) for x in v_tree[b][u][g]])
                qv = [float(x) for x in q[b][i][h]]
                s = [scale * sum(qv[d] * kk[d] for d in range(D)) for kk in keys]
                mx = max(s)
                w = [math.exp(x - mx) for x in s]
                tot = sum(w)
                oi.append([sum(w[t] * vals[t][d] for t in range(len(w))) / tot
                           for d in range(D)])
            ob.append(oi)
        out.append(ob)
    return out


def argmax_first(row):
    best_i, best_v = 0, float(row[0])
    for i in range(1, len(row)):
        if float(row[i]) > best_v:
            best_i, best_v = i, float(row[i])
    return best_i


def accept(logits, draft_tok, parent, Dmax):
    """Returns (accept_len list, path lists, tgt lists)."""
    B = len(parent)
    lens, paths, tgts = [], [], []
    for b in range(B):
        par = [int(x) for x in parent[b]]
        N = len(par)
        tgt = [argmax_first(logits[b][i]) for i in range(N)]
        tgts.append(tgt)
        if not _valid_tree(par):
            lens.append(-1)
            paths.append([-1] * Dmax)
            continue
        best = None
        for v in range(N):
            pth = _root_path(par, v)
            if all(int(draft_tok[b][pth[t]]) == tgt[pth[t - 1]]
                   for t in range(1, len(pth))):
                if best is None or len(pth) > len(best):
                    best = pth
        if len(best) > Dmax:
            lens.append(-1)
            paths.append([-1] * Dmax)
        else:
            lens.append(len(best))
            paths.append(best + [-1] * (Dmax - len(best)))
    return lens, paths, tgts


def topw(logits_row, W):
    """Pure-Python top-W of one row: tokens by (value desc, index asc) and
    their log-probabilities from an exactly summed log-sum-exp."""
    xs = [float(x) for x in logits_row]
    m = max(xs)
    lse = m + math.log(math.fsum(math.exp(x - m) for x in xs))
    order = sorted(range(len(xs)), key=lambda i: (-xs[i], i))[:W]
    return order, [xs[i] - lse for i in order]


def tree_in_score_order(tok, logp, budget):
    """The tree of best-first expansion without a priority queue, for one
    sequence whose accumulated scores are all distinct and whose
    log-probabilities are negative.

    Every node of the full W-ary tree of depth Nd has a fixed score (float32
    accumulation along its path).  Because a child scores below its parent,
    best-first pops nodes in plain descending score order; each popped node
    above the maximum depth appends its W children in candidate order until
    the budget is reached.  Returns (parent, token, depth, score) lists.
    """
    Nd, W = len(tok), len(tok[0])
    f32 = np.float32
    # all nodes of the full tree, keyed by their path of candidate ranks
    full = {(): f32(0.0)}
    frontier = [()]
    for d in range(Nd):
        nxt = []
        for p in frontier:
            for k in range(W):
                full[p + (k,)] = f32(full[p] + f32(logp[d][k]))
                nxt.append(p + (k,))
        frontier = nxt
    order = sorted((p for p in full if len(p) < Nd), key=lambda p: -float(full[p]))
    index = {(): 0}
    parent, token, depth, score = [-1], [-1], [0], [f32(0.0)]
    for p in order:
        if len(parent) == budget:
            break
        if p not in index:      # not added: the budget ran out before it
            break
        for k in range(W):
            if len(parent) == budget:
                break
            c = p + (k,)
            index[c] = len(parent)
            parent.append(index[p])
            token.append(int(tok[len(p)][k]))
            depth.append(len(c))
            score.append(full[c])
    return parent, token, depth, score


def commit_tail_in_place(cache, path, accept_len, kv_len):
    """Tree-tail commit done in place, one row at a time in increasing
    order: row kv_len + j takes row kv_len + path[j].  Correct because a
    root-to-node path has path[j] >= j (a node's index exceeds its depth),
    so no row is read after it was overwritten."""
    c = [[row.copy() for row in seq] for seq in np.asarray(cache)]
    for b in range(len(c)):
        n = int(accept_len[b])
        if n < 1:
            continue
        kl = int(kv_len[b])
        for j in range(n):
            c[b][kl + j] = c[b][kl + int(path[b][j])].copy()
    return np.array(c)


def block_causal(q, k_ctx, v_ctx, k_blk, v_blk, anchors, scale=None):
    """Training-mask attention with Python loops: query (b, k, j, h) sees
    context rows t < anchor and block k's positions 0..j."""
    B, A, S, Hq, D = np.asarray(q).shape
    L, Hkv = np.asarray(k_ctx).shape[1:3]
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    out = np.zeros((B, A, S, Hq, D))
    for b in range(B):
        for k in range(A):
            a = min(max(int(anchors[b][k]), 0), L)
            for j in range(S):
                for h in range(Hq):
                    g = h // G
                    keys = [(k_ctx[b][t][g], v_ctx[b][t][g]) for t in range(a)]
                    keys += [(k_blk[b][k][i][g], v_blk[b][k][i][g]) for i in range(j + 1)]
                    sc = [scale * sum(float(x) * float(y) for x, y in zip(q[b][k][j][h], kk))
                          for kk, _ in keys]
                    mx = max(sc)
                    w = [math.exp(x - mx) for x in sc]
                    tot = sum(w)
                    for d in range(D):
                        out[b, k, j, h, d] = sum(wi * float(vv[d]) for wi, (_, vv) in
                                                 zip(w, keys)) / tot
    return out


def _softmax_list(row, T):
    m = max(float(x) / T for x in row)
    e = [math.exp(float(x) / T - m) for x in row]
    s = sum(e)
    return [x / s for x in e]


def accept_sampled(logits, draft_tok, parent, u_accept, seed, T, Dmax):
    """Sampled tree acceptance, checked path by path: a node is taken from
    its parent when its own test passes and no earlier sibling's does (each
    sibling's test against the mass its earlier siblings' distinct tokens
    left, in Python floats); the result is the longest root-to-node path made
    only of taken nodes.  The correction token by a Python-loop exponential
    race over scalar Philox words, with the end node's child tokens removed."""
    from .philox import philox4x32, uniform_open
    B, N = len(parent), len(parent[0])
    V = len(logits[0][0])
    out_len, out_path, out_corr = [], [], []
    for b in range(B):
        par = [int(x) for x in parent[b]]
        if not _valid_tree(par):
            out_len.append(-1); out_path.append([-1] * Dmax); out_corr.append(-1)
            continue
        probs = [_softmax_list(logits[b][v], T) for v in range(N)]
        passes = [False] * N
        for c in range(1, N):
            sibs = [j for j in range(1, c) if par[j] == par[c]]
            seen, mass = [], 0.0
            for j in sibs:
                yj = int(draft_tok[b][j])
                if 0 <= yj < V and yj not in seen:
                    seen.append(yj)
                    mass += probs[par[c]][yj]
            y = int(draft_tok[b][c])
            e = probs[par[c]][y] if 0 <= y < V and y not in seen else 0.0
            passes[c] = float(u_accept[b][c]) * (1.0 - mass) < e
        taken = [c > 0 and passes[c] and not any(passes[j] for j in range(1, c)
                                                  if par[j] == par[c]) for c in range(N)]
        best = [0]
        for i in range(1, N):
            pth = _root_path(par, i)
            if all(taken[x] for x in pth[1:]) and len(pth) > len(best):
                best = pth
        if len(best) > Dmax:
            out_len.append(-1); out_path.append([-1] * Dmax); out_corr.append(-1)
            continue
        end = best[-1]
        kids = {int(draft_tok[b][c]) for c in range(1, N) if par[c] == end}
        w = [0.0 if x in kids else probs[end][x] for x in range(V)]
        if not any(x > 0 for x in w):
            w = probs[end]
        tok, top = -1, -1.0
        for x in range(V):
            word = philox4x32((x // 4, b, 0, 0), (seed & 0xFFFFFFFF, seed >> 32))[x % 4]
            race = w[x] / -math.log(uniform_open(word)) if w[x] > 0 else -1.0
            if race > top:
                tok, top = x, race
        out_len.append(len(best))
        out_path.append(best + [-1] * (Dmax - len(best)))
        out_corr.append(tok)
    return np.array(out_len), np.array(out_path), np.array(out_corr)
