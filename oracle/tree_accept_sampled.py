"""Oracle of non-greedy (temperature T > 0) tree acceptance (test
infrastructure only).

What it computes (Sec. 2.4, tree verification with the speculative sampling
rule; the T = 1 rows of the results tables):

  * target distribution at node v: p_v = softmax(logits[v] / T), the target's
    next-token distribution after the context plus v's root path;
  * draft distribution of depth d: q_d = softmax(draft_logits[d - 1] / T),
    the draft head's distribution for the token at depth d (the parallel
    head's distributions are position-wise, as in tree drafting);
  * draft node i (token y_i, parent u, depth d) passes its test when
    u_i < min(1, p_u(y_i) / q_d(y_i)), i.e. u_i * q_d(y_i) < p_u(y_i), with
    u_i the node's uniform random number; it is accepted when it passes and
    its parent is accepted (the root is always accepted);
  * the result is the deepest accepted node v and its root path;
  * the correction token is drawn at v: from the residual
    max(0, p_v - q_{d(v)+1}) (normalised) when v has children, all of which
    were rejected; from p_v when v is a leaf (no draft was offered there).

Readings where the paper is silent:
  * each node has one uniform, shared by every branch through it, so one
    acceptance test per node and the deepest accepted node decides, as in
    the greedy rule (lowest node index among equally deep ones);
  * the temperature scales target and draft logits alike;
  * the residual of a node whose children were all rejected uses the single
    draft distribution of their depth; an all-zero residual (p = q) falls
    back to p_v;
  * sampling a token from weights w uses the exponential race
    argmax_x w(x) / E_x with E_x = -ln U(b, x) (equivalently Gumbel-max), ties
    to the lowest index, where U(b, x) is word x mod 4 of
    Philox4x32-10(counter = (x div 4, b, 0, 0), key = (seed low, seed high))
    mapped to (0, 1) by its top 23 bits, ((word >> 9) + 1/2) / 2^23, a value
    exact in fp32;
  * a tree deeper than the draft logits, an invalid tree or a path longer
    than Dmax give accept_len = -1, path all -1 and correction -1.
"""
from __future__ import annotations

import numpy as np

from .philox import philox4x32_array
from .tree_attention import tree_structure


def _softmax(x: np.ndarray) -> np.ndarray:
    z = x - x.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=-1, keepdims=True)


def race_uniforms(b: int, V: int, seed: int) -> np.ndarray:
    """U(b, x) for x in [0, V) as float64."""
    n4 = (V + 3) // 4
    ctr = np.arange(n4, dtype=np.uint64)
    out = philox4x32_array(ctr, np.full(n4, b), np.zeros(n4), np.zeros(n4),
                           seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    words = np.stack(out, axis=1).reshape(-1)[:V]
    return ((words >> np.uint64(9)).astype(np.float64) + 0.5) / 8388608.0


def race_sample(w: np.ndarray, b: int, seed: int):
    """Exponential race over weights w >= 0: (token, relative gap between the
    best and second-best race values (inf when only one is positive), the
    second-best token)."""
    e = -np.log(race_uniforms(b, len(w), seed))
    score = np.where(w > 0, w / e, -1.0)
    tok = int(np.argmax(score))
    top = score[tok]
    rest = score.copy()
    rest[tok] = -1.0
    runner = int(np.argmax(rest))
    second = rest[runner]
    gap = np.inf if second <= 0 else (top - second) / top
    return tok, gap, runner


def tree_accept_sampled(logits, draft_logits, draft_tok, parent, u_accept, seed: int,
                        temperature: float, Dmax: int, detail: bool = False):
    """logits [B, N, V], draft_logits [B, Nd, V], draft_tok/parent [B, N],
    u_accept [B, N].  Returns (accept_len [B], path [B, Dmax],
    correction [B]) as int32, and with detail=True a dict of per-node test
    margins (|p - u q| relative to max(p, q)), the sampling gap and the
    second-best token of each sequence's race."""
    lg = np.asarray(logits, dtype=np.float64)
    dl = np.asarray(draft_logits, dtype=np.float64)
    B, N, V = lg.shape
    Nd = dl.shape[1]
    T = float(temperature)
    accept_len = np.full(B, -1, dtype=np.int32)
    path = np.full((B, Dmax), -1, dtype=np.int32)
    corr = np.full(B, -1, dtype=np.int32)
    margin = np.full((B, N), np.inf)
    gaps = np.full(B, np.inf)
    runner = np.full(B, -1, dtype=np.int32)
    for b in range(B):
        valid, _, depth = tree_structure(parent[b])
        if not valid or depth.max() > Nd:
            continue
        p = _softmax(lg[b] / T)               # [N, V]: next-token distribution at each node
        q = _softmax(dl[b] / T)               # [Nd, V]: row d - 1 is depth d
        acc = np.zeros(N, dtype=bool)
        acc[0] = True
        for i in range(1, N):
            u, d, y = int(parent[b, i]), int(depth[i]), int(draft_tok[b, i])
            pi, qi = p[u, y], q[d - 1, y]
            test = float(u_accept[b, i]) * qi < pi
            margin[b, i] = abs(pi - float(u_accept[b, i]) * qi) / max(pi, qi, 1e-300)
            acc[i] = acc[u] and test
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
        path[b, :length] = walk[::-1]
        accept_len[b] = length
        has_child = bool(np.any(np.asarray(parent[b])[1:] == best))
        w = np.maximum(p[best] - q[depth[best]], 0.0) if has_child else p[best]
        if not np.any(w > 0):
            w = p[best]
        corr[b], gaps[b], runner[b] = race_sample(w, b, seed)
    if detail:
        return accept_len, path, corr, {"margin": margin, "gap": gaps, "runner_up": runner}
    return accept_len, path, corr
