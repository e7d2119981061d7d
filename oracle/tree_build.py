"""Oracle of budgeted tree drafting (test infrastructure only).

What it computes (Sec. 2.4, "Parallel Tree Drafting"; App. "Tree-Drafting
Algorithm Details", Alg. 1; App. "vLLM Implementation Details"):

  draft_topw   one draft-head pass gives a distribution for every draft
               depth; the W most likely tokens of each depth, with their log
               probabilities, are the candidate children of every node one
               depth above.
  build_tree   best-first expansion under a node budget: a priority queue
               of nodes ordered by the accumulated draft log-probability of
               their root path (the paper's default score); the best node is
               popped and, unless it sits at the maximum draft depth, gets up
               to W children (the candidates of the next depth, in order),
               each pushed with its own score, until the tree holds `budget`
               nodes or the queue is empty.

Readings where the paper is silent:
  * the root (node 0, depth 0, score 0) is the already-sampled token; the
    budget counts it;
  * the candidates of depth d+1 are the same for every node at depth d (the
    position-wise distributions of the parallel head), visited in
    decreasing log-probability, equal values by lower token id;
  * equal scores pop the lower node index first (node index = insertion
    order);
  * scores accumulate in float32, child = float32(parent + log-prob): the
    kernel's precision, because these comparisons decide the tree;
  * log-probabilities themselves are exact (float64 log-softmax) here.
"""
from __future__ import annotations

import heapq

import numpy as np


def draft_topw(logits: np.ndarray, W: int):
    """logits [..., V] -> (tok [..., W] int64, logp [..., W] float64).

    logp = logits - logsumexp(logits) in float64; tokens are the W largest
    logits, ties by lower index (log-softmax is monotone, so these are also
    the W most likely tokens).
    """
    x = np.asarray(logits, dtype=np.float64)
    V = x.shape[-1]
    if not 1 <= W <= V:
        raise ValueError("need 1 <= W <= V")
    m = x.max(axis=-1, keepdims=True)
    lse = m + np.log(np.exp(x - m).sum(axis=-1, keepdims=True))
    order = np.argsort(-x, axis=-1, kind="stable")[..., :W]
    tok = order.astype(np.int64)
    logp = np.take_along_axis(x, order, axis=-1) - lse
    return tok, logp


def build_tree(tok: np.ndarray, logp: np.ndarray, budget: int, root_tok=None):
    """Alg. 1 for each sequence.

    tok, logp: [B, Nd, W] candidates per draft depth (Nd = maximum draft
    depth); logp is taken as float32.  Returns dict of
      parent [B, budget] int64 (-1 for the root and unused slots),
      token  [B, budget] int64 (root_tok[b] or -1 at the root, -1 unused),
      depth  [B, budget] int64 (-1 unused),
      score  [B, budget] float32 (-inf unused),
      n_nodes [B] int64.
    """
    tok = np.asarray(tok)
    lp32 = np.asarray(logp, dtype=np.float32)
    B, Nd, W = tok.shape
    if budget < 1:
        raise ValueError("budget >= 1")
    parent = np.full((B, budget), -1, dtype=np.int64)
    token = np.full((B, budget), -1, dtype=np.int64)
    depth = np.full((B, budget), -1, dtype=np.int64)
    score = np.full((B, budget), -np.inf, dtype=np.float32)
    n_nodes = np.zeros(B, dtype=np.int64)
    for b in range(B):
        token[b, 0] = -1 if root_tok is None else int(root_tok[b])
        depth[b, 0] = 0
        score[b, 0] = np.float32(0.0)
        n = 1
        # max-heap on score, lower node index first on equal scores
        heap = [(-np.float32(0.0), 0)]
        while n < budget and heap:
            _, v = heapq.heappop(heap)
            d = int(depth[b, v])
            if d == Nd:
                continue
            for k in range(W):
                if n == budget:
                    break
                s = np.float32(score[b, v] + lp32[b, d, k])
                parent[b, n], token[b, n], depth[b, n], score[b, n] = v, tok[b, d, k], d + 1, s
                heapq.heappush(heap, (-s, n))
                n += 1
        n_nodes[b] = n
    return {"parent": parent, "token": token, "depth": depth, "score": score, "n_nodes": n_nodes}
