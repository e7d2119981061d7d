"""Oracle of non-greedy (temperature T > 0) tree acceptance (test
infrastructure only: nothing on the product path imports it).

What it computes.  Sec. 2.4 verifies a tree with the speculative sampling
rule (eq. nongreedy_specdec: a draft token y is accepted with probability
min(1, p(y) / q(y)), a correction token is drawn from the target when a draft
is rejected) and Sec. 2.2 / Sec. 3.4 state that verification is lossless:
the emitted tokens follow the target distribution.  The tree's children are
not draws from q: Alg. 1 and App. E expand a node with the top-W draft
tokens of the next depth, a deterministic choice.  The proposal that produced
such a child is the point mass at its token, so the acceptance rule of
eq. nongreedy_specdec with that proposal, applied to a node's children one
after another against the target distribution left over by the rejected
ones (multi-candidate speculative sampling), is the reading that keeps
verification lossless:

  * p_v = softmax(logits[v] / T): the target's next-token distribution after
    the context and v's root path;
  * the walk starts at the root (always accepted).  At the current node v
    its children c are tested in increasing index order.  With R the set of
    tokens of v's children rejected so far and S = sum of p_v over R, child c
    (token y_c) passes when u_c * (1 - S) < e_c, where e_c = p_v(y_c) if y_c
    is a valid token not in R and e_c = 0 otherwise; that is
    u_c < min(1, p'(y_c)) for the renormalised residual p' = p_v without R.
    The first child that passes becomes the current node; a child that fails
    adds y_c to R.  The walk stops at a node none of whose children passes;
    it is the last node of the path.
  * the correction token is drawn at the last node v from the final residual:
    p_v with every token of v's children removed (all of them were tested
    and rejected), renormalised; from p_v itself when v is a leaf.

With u_c uniform on [0, 1), child c is reached and accepted with
probability e_c (the residual's mass before it, times e_c over that mass), so
the walk ends at node v with probability (product of p over v's root path) x
(1 - sum of p_v over the distinct tokens of v's children), and the first
emitted token (a child's token, or the correction) is distributed exactly as
p at the root.

Readings where the paper is silent:
  * the temperature scales the target logits; the draft probabilities do not
    enter the rule (a deterministic child's proposal is its point mass);
  * a repeated token among a node's children is never accepted after its
    first occurrence was rejected (its residual mass is zero), and a token
    outside [0, V) never passes;
  * a residual with no mass left (possible only through rounding) falls back
    to p_v for the correction;
  * sampling a token from weights w uses the exponential race
    argmax_x w(x) / E_x with E_x = -ln U(b, x) (equivalently Gumbel-max), ties
    to the lowest index, where U(b, x) is word x mod 4 of
    Philox4x32-10(counter = (x div 4, b, 0, 0), key = (seed low, seed high))
    mapped to (0, 1) by its top 23 bits, ((word >> 9) + 1/2) / 2^23, a value
    exact in fp32;
  * an invalid tree or a path longer than Dmax gives accept_len = -1, path
    all -1 and correction -1.
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


def tree_accept_sampled(logits, draft_tok, parent, u_accept, seed: int, temperature: float,
                        Dmax: int, detail: bool = False):
    """logits [B, N, V], draft_tok/parent [B, N], u_accept [B, N].  Returns
    (accept_len [B], path [B, Dmax], correction [B]) as int32, and with
    detail=True a dict of per-node test margins (|e - u (1 - S)| relative to
    max(e, u (1 - S)), inf for nodes never tested), the sampling gap and the
    second-best token of each sequence's race."""
    lg = np.asarray(logits, dtype=np.float64)
    B, N, V = lg.shape
    T = float(temperature)
    accept_len = np.full(B, -1, dtype=np.int32)
    path = np.full((B, Dmax), -1, dtype=np.int32)
    corr = np.full(B, -1, dtype=np.int32)
    margin = np.full((B, N), np.inf)
    gaps = np.full(B, np.inf)
    runner = np.full(B, -1, dtype=np.int32)
    for b in range(B):
        par = np.asarray(parent[b])
        valid, _, depth = tree_structure(par)
        if not valid:
            continue
        p = _softmax(lg[b] / T)               # [N, V]: next-token distribution at each node
        walk = [0]
        rejected = set()
        while True:
            v = walk[-1]
            rejected = set()
            S = 0.0
            nxt = None
            for c in range(v + 1, N):       # children follow their parent
                if par[c] != v:
                    continue
                y = int(draft_tok[b, c])
                ok_tok = 0 <= y < V and y not in rejected
                e = p[v, y] if ok_tok else 0.0
                lhs = float(u_accept[b, c]) * (1.0 - S)
                margin[b, c] = abs(e - lhs) / max(e, lhs, 1e-300)
                if lhs < e:
                    nxt = c
                    break
                if ok_tok:
                    rejected.add(y)
                    S += e
            if nxt is None:
                break
            walk.append(nxt)
        v = walk[-1]
        if len(walk) > Dmax:
            continue
        path[b, :len(walk)] = walk
        accept_len[b] = len(walk)
        w = p[v].copy()
        if rejected:
            w[sorted(rejected)] = 0.0
        if not np.any(w > 0):
            w = p[v]
        corr[b], gaps[b], runner[b] = race_sample(w, b, seed)
        assert len(walk) == depth[v] + 1
    if detail:
        return accept_len, path, corr, {"margin": margin, "gap": gaps, "runner_up": runner}
    return accept_len, path, corr
