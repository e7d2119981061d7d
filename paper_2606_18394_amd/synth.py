"""Seeded synthetic inputs for tree verification.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic (no attention, no argmax, no acceptance).  Both the HIP
path's tests/bench and the CPU oracle consume what it produces.

Workloads follow the shapes of the paper's targets (Qwen3-8B, Qwen3-30B-A3B,
Qwen3-32B attention shapes; Sec. 3.1 and App. D give the 32/8-head, D=128
geometry) with draft trees as produced by budgeted tree drafting (Sec. 2.4,
Alg. 1: node budget, maximum depth, branching width; node 0 is the root,
App. E).  Every node's parent precedes it, as in Alg. 1 where a child is
appended after its parent.

bf16 tensors are returned as ``uint16`` bit patterns obtained from float32
draws by round-to-nearest-even.
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Optional, Tuple

import numpy as np

# Cache rows at or beyond a sequence's kv_len are filled with this value so a
# kernel that lets them leak into a result fails loudly.  1000.0 is exact in
# bf16 (0x447A).
POISON_BF16 = np.uint16(0x447A)


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    D: int
    L: int            # padded cache length Lmax
    N: int            # tree nodes per sequence, root included
    depth: int        # depth cap (root at depth 0)
    branching: Optional[int]   # max children per node, None = unlimited
    spine: bool       # force a chain 0-1-...-depth so the max depth is exact
    ragged: Optional[Tuple[int, int]]  # kv_len ~ U[lo, hi] inclusive, else all L
    V: int
    logits_dtype: str  # "f32" or "bf16"
    logit_std: float
    p_match: float     # P(draft token = target argmax at the parent)
    seed: int

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def Dmax(self) -> int:
        return self.depth + 1


WORKLOADS = {
    "tiny": Workload("tiny", B=1, Hq=4, Hkv=2, D=64, L=256, N=16, depth=4,
                     branching=None, spine=False, ragged=None, V=1024,
                     logits_dtype="f32", logit_std=1.0, p_match=0.5, seed=0),
    "qwen3_8b": Workload("qwen3_8b", B=1, Hq=32, Hkv=8, D=128, L=4096, N=64,
                         depth=8, branching=4, spine=True, ragged=None,
                         V=151936, logits_dtype="bf16", logit_std=2.0,
                         p_match=0.6, seed=1),
    "long_ctx": Workload("long_ctx", B=1, Hq=32, Hkv=8, D=128, L=32768, N=128,
                         depth=12, branching=4, spine=True, ragged=None,
                         V=151936, logits_dtype="bf16", logit_std=2.0,
                         p_match=0.6, seed=2),
    "batched_30b_a3b": Workload("batched_30b_a3b", B=16, Hq=32, Hkv=4, D=128,
                                L=16384, N=64, depth=8, branching=4,
                                spine=False, ragged=(1024, 16384), V=151936,
                                logits_dtype="bf16", logit_std=2.0,
                                p_match=0.5, seed=3),
    "big_tree_32b": Workload("big_tree_32b", B=1, Hq=64, Hkv=8, D=128, L=8192,
                             N=512, depth=16, branching=8, spine=True,
                             ragged=None, V=151936, logits_dtype="bf16",
                             logit_std=2.0, p_match=0.7, seed=4),
}

WORKLOAD_ORDER = ["tiny", "qwen3_8b", "long_ctx", "batched_30b_a3b", "big_tree_32b"]


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit pattern, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def random_tree(rng: np.random.Generator, N: int, depth: int,
                branching: Optional[int] = None, spine: bool = False) -> np.ndarray:
    """Parent array of a random rooted tree in topological order.

    Node i > 0 picks its parent uniformly among earlier nodes that are below
    the depth cap and still have room for a child.  With ``spine`` the nodes
    1..depth form a chain first so the maximum depth is exactly ``depth``.
    """
    parent = np.full(N, -1, dtype=np.int32)
    dep = np.zeros(N, dtype=np.int64)
    nchild = np.zeros(N, dtype=np.int64)
    for i in range(1, N):
        if spine and i <= depth:
            p = i - 1
        else:
            ok = dep[:i] < depth
            if branching is not None:
                ok &= nchild[:i] < branching
            cand = np.flatnonzero(ok)
            if cand.size == 0:
                raise ValueError("tree caps leave no room for node %d" % i)
            p = int(cand[rng.integers(0, cand.size)])
        parent[i] = p
        dep[i] = dep[p] + 1
        nchild[p] += 1
    return parent


def chain_tree(N: int) -> np.ndarray:
    return np.arange(-1, N - 1, dtype=np.int32)


def star_tree(N: int) -> np.ndarray:
    p = np.zeros(N, dtype=np.int32)
    p[0] = -1
    return p


def _normal_bf16(rng: np.random.Generator, shape, std: float = 1.0) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return bf16_bits(x)


def make_inputs(rng: np.random.Generator, *, B: int, N: int, Hq: int, Hkv: int,
                D: int, Lmax: int, V: int, trees: np.ndarray,
                kv_len: np.ndarray, logits_dtype: str = "bf16",
                logit_std: float = 1.0, p_match: float = 0.5,
                poison: bool = True, with_logits: bool = True) -> dict:
    """Draw q/k/v, logits and the draft-token randomness for given trees.

    Draw order after the trees and kv_len: q, k_cache, v_cache, k_tree,
    v_tree, logits, match flags, random tokens.
    """
    trees = np.ascontiguousarray(trees, dtype=np.int32).reshape(B, N)
    kv_len = np.ascontiguousarray(kv_len, dtype=np.int32).reshape(B)
    inp = {
        "B": B, "N": N, "Hq": Hq, "Hkv": Hkv, "D": D, "Lmax": Lmax, "V": V,
        "parent": trees, "kv_len": kv_len,
        "q": _normal_bf16(rng, (B, N, Hq, D)),
        "k_cache": _normal_bf16(rng, (B, Lmax, Hkv, D)),
        "v_cache": _normal_bf16(rng, (B, Lmax, Hkv, D)),
        "k_tree": _normal_bf16(rng, (B, N, Hkv, D)),
        "v_tree": _normal_bf16(rng, (B, N, Hkv, D)),
    }
    if poison:
        for b in range(B):
            inp["k_cache"][b, kv_len[b]:] = POISON_BF16
            inp["v_cache"][b, kv_len[b]:] = POISON_BF16
    if with_logits:
        if logits_dtype == "f32":
            lg = rng.standard_normal(size=(B, N, V), dtype=np.float32)
            if logit_std != 1.0:
                lg *= np.float32(logit_std)
            inp["logits"] = lg
        elif logits_dtype == "bf16":
            inp["logits"] = _normal_bf16(rng, (B, N, V), logit_std)
        else:
            raise ValueError(logits_dtype)
        inp["logits_dtype"] = logits_dtype
        inp["match"] = rng.random(size=(B, N)) < p_match
        inp["rand_tok"] = rng.integers(0, V, size=(B, N), dtype=np.int32)
    return inp


def draw(w: Workload, seed: Optional[int] = None, with_logits: bool = True,
         poison: bool = True) -> dict:
    """All inputs of a named workload (trees, kv_len, tensors, draft randomness)."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    trees = np.stack([random_tree(rng, w.N, w.depth, w.branching, w.spine)
                      for _ in range(w.B)])
    if w.ragged is not None:
        lo, hi = w.ragged
        kv_len = rng.integers(lo, hi + 1, size=w.B).astype(np.int32)
    else:
        kv_len = np.full(w.B, w.L, dtype=np.int32)
    inp = make_inputs(rng, B=w.B, N=w.N, Hq=w.Hq, Hkv=w.Hkv, D=w.D, Lmax=w.L,
                      V=w.V, trees=trees, kv_len=kv_len,
                      logits_dtype=w.logits_dtype, logit_std=w.logit_std,
                      p_match=w.p_match, poison=poison, with_logits=with_logits)
    inp["workload"] = w.name
    inp["Dmax"] = w.Dmax
    return inp


def draft_tokens(parent: np.ndarray, tgt: np.ndarray, match: np.ndarray,
                 rand_tok: np.ndarray) -> np.ndarray:
    """Assemble draft tokens: node i copies ``tgt`` at its parent where
    ``match`` is set, else takes its random token.  The root keeps its random
    token (it is ignored by verification).  ``tgt`` is supplied by the caller.
    """
    parent = np.asarray(parent)
    B, N = parent.shape
    out = np.array(rand_tok, dtype=np.int32, copy=True)
    for b in range(B):
        for i in range(1, N):
            if match[b, i]:
                out[b, i] = tgt[b, parent[b, i]]
    return out


def draft_width(w: Workload) -> int:
    """Branching width W of the workload's tree drafting: its branching cap,
    4 where the tree is uncapped."""
    return w.branching if w.branching else 4


def draft_logits(w: Workload, seed: Optional[int] = None) -> np.ndarray:
    """Draft-head logits [B, depth, V] (one row per draft depth) for the
    workload's tree drafting, drawn like its target logits (same std and
    dtype: bf16 bit patterns, or float32) from a stream of their own."""
    rng = np.random.default_rng(1000 + (w.seed if seed is None else seed))
    x = (rng.standard_normal((w.B, w.depth, w.V), dtype=np.float32) * np.float32(w.logit_std))
    return x if w.logits_dtype == "f32" else bf16_bits(x)


def with_shape(w: Workload, **kw) -> Workload:
    return replace(w, **kw)


def block_table(rng: np.random.Generator, B: int, max_blocks: int, spare: int = 0,
                used=None) -> Tuple[np.ndarray, int]:
    """A shuffled paged-cache block table: every sequence gets max_blocks
    distinct pool blocks drawn from a pool of B * max_blocks + spare blocks.
    With ``used`` ([B] block counts), entries past a sequence's used blocks
    are -1 (unallocated).  Returns (table [B, max_blocks] int32, num_blocks)."""
    num_blocks = B * max_blocks + spare
    bt = rng.permutation(num_blocks)[:B * max_blocks].astype(np.int32).reshape(B, max_blocks)
    if used is not None:
        for b in range(B):
            bt[b, int(used[b]):] = -1
    return bt, num_blocks


def scatter_pool(rng: np.random.Generator, cache: np.ndarray, bt: np.ndarray, num_blocks: int,
                 block_size: int) -> np.ndarray:
    """Lay a contiguous cache [B, Lmax, ...] out as a pool [num_blocks,
    block_size, ...]: rows j*block_size.. of sequence b go to block bt[b, j]
    (entries < 0 are skipped, as are rows past Lmax).  Blocks no sequence
    owns hold random bf16 values."""
    B, Lmax = cache.shape[:2]
    pool = _normal_bf16(rng, (num_blocks, block_size) + cache.shape[2:])
    for b in range(B):
        for j in range(bt.shape[1]):
            lo = j * block_size
            if bt[b, j] < 0 or lo >= Lmax:
                continue
            hi = min(lo + block_size, Lmax)
            pool[bt[b, j], :hi - lo] = cache[b, lo:hi]
    return pool
