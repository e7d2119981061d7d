"""Thin ctypes binding of libtreeverify.so.

Argument marshalling only: torch tensors serve as device buffers and the
current torch stream as the HIP stream; every step of the computation runs in
the library's HIP kernels.  There is no fallback: if the library is missing
or the tensors are not on a GPU, the calls raise.
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtreeverify.so")

TV_BF16, TV_F32 = 0, 1
MAX_NODES = 2048

_lib = None
_lock = threading.Lock()
_workspaces = {}


def load_library() -> ctypes.CDLL:
    """Load the built library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                "libtreeverify.so is not built (run __graft_entry__.build() or "
                "python paper_2606_18394_amd/build.py)")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i32p, ci, sz = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        lib.tv_status_string.restype = ctypes.c_char_p
        lib.tv_status_string.argtypes = [ci]
        lib.tv_version.restype = ci
        lib.tv_version.argtypes = []
        lib.tv_tree_verify_attention_workspace.restype = sz
        lib.tv_tree_verify_attention_workspace.argtypes = [ci] * 6
        lib.tv_tree_verify_attention.restype = ci
        lib.tv_tree_verify_attention.argtypes = (
            [vp] * 5 + [i32p, i32p, vp] + [ci] * 6 + [ctypes.c_float, vp, sz, vp])
        lib.tv_tree_accept_workspace.restype = sz
        lib.tv_tree_accept_workspace.argtypes = [ci] * 3
        lib.tv_tree_accept.restype = ci
        lib.tv_tree_accept.argtypes = (
            [vp, ci, i32p, i32p] + [ci] * 4 + [i32p, i32p, i32p, vp, sz, vp])
        lib.tv_tree_accept_noalloc.restype = ci
        lib.tv_tree_accept_noalloc.argtypes = [vp, ci, i32p, i32p] + [ci] * 4 + [i32p] * 3 + [vp]
        lib.tv_draft_topw_workspace.restype = sz
        lib.tv_draft_topw_workspace.argtypes = [ci] * 3
        lib.tv_draft_topw.restype = ci
        lib.tv_draft_topw.argtypes = [vp] + [ci] * 5 + [i32p, vp, vp, sz, vp]
        lib.tv_build_tree.restype = ci
        lib.tv_build_tree.argtypes = [i32p, vp, i32p] + [ci] * 4 + [i32p, i32p, i32p, vp, i32p, vp]
        lib.tv_tree_verify_attention_paged.restype = ci
        lib.tv_tree_verify_attention_paged.argtypes = (
            [vp, vp, vp, i32p] + [ci] * 3 + [vp, vp, i32p, i32p, vp] + [ci] * 5
            + [ctypes.c_float, vp, sz, vp])
        lib.tv_block_causal_attention_workspace.restype = sz
        lib.tv_block_causal_attention_workspace.argtypes = [ci] * 7
        lib.tv_block_causal_attention.restype = ci
        lib.tv_block_causal_attention.argtypes = (
            [vp] * 5 + [i32p, vp] + [ci] * 7 + [ctypes.c_float, vp, sz, vp])
        lib.tv_tree_accept_sampled_workspace.restype = sz
        lib.tv_tree_accept_sampled_workspace.argtypes = [ci] * 3
        lib.tv_tree_accept_sampled.restype = ci
        lib.tv_tree_accept_sampled.argtypes = (
            [vp, ci, i32p, i32p, vp, ctypes.c_ulonglong, ctypes.c_float] + [ci] * 4
            + [i32p, i32p, i32p, vp, sz, vp])
        lib.tv_commit_path.restype = ci
        lib.tv_commit_path.argtypes = [vp, vp, i32p, i32p, vp, vp, i32p] + [ci] * 6 + [vp]
        lib.tv_commit_path_paged.restype = ci
        lib.tv_commit_path_paged.argtypes = (
            [vp, vp, i32p, i32p, vp, vp, i32p] + [ci] * 3 + [i32p] + [ci] * 5 + [vp])
        _lib = lib
        return lib


def status_string(rc: int) -> str:
    return load_library().tv_status_string(rc).decode()


def _check(rc: int) -> None:
    if rc != 0:
        raise RuntimeError(status_string(rc))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _need(t, name, dtype, shape=None, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _need_tree(k_tree, v_tree, shape, device):
    """Tree K/V tensors, or both None (tree-tail layout)."""
    if (k_tree is None) != (v_tree is None):
        raise ValueError("k_tree and v_tree must both be given or both be None")
    if k_tree is not None:
        _need(k_tree, "k_tree", torch.bfloat16, shape, device)
        _need(v_tree, "v_tree", torch.bfloat16, shape, device)


_retired = []


def workspace(kind: str, nbytes: int, device, stream_ptr: int) -> torch.Tensor:
    """Zero-filled workspace cached per (kind, device, stream); grows as needed.

    A HIP graph captured with a cached workspace keeps writing to that
    buffer's address on every replay, so a workspace that a larger call
    replaces is kept alive (in ``_retired``) rather than freed: its memory is
    never handed to another tensor while the process runs.  Under stream
    capture nothing is allocated: the cached workspace must already be large
    enough (make one eager call of the same or a larger size on the capturing
    stream first), or the caller passes ``workspace_tensor``.
    """
    key = (kind, str(device), stream_ptr)
    ws = _workspaces.get(key)
    if ws is None or ws.numel() < nbytes:
        if torch.device(device).type == "cuda" and torch.cuda.is_current_stream_capturing():
            raise RuntimeError(
                f"the cached {kind} workspace of this stream is missing or smaller than the "
                f"{nbytes} bytes this call needs, and a workspace cannot be allocated during "
                f"graph capture: call once eagerly on the capturing stream first, or pass "
                f"workspace_tensor")
        if ws is not None:
            _retired.append(ws)
        ws = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=device)
        _workspaces[key] = ws
    return ws


def tree_verify_attention(q, k_cache, v_cache, k_tree, v_tree, parent, out,
                          kv_len=None, scale=None, workspace_tensor=None):
    """out[b,i,h] = tree-masked attention of node i (bf16 in, bf16 out).

    q [B,N,Hq,D], k_cache/v_cache [B,Lmax,Hkv,D], k_tree/v_tree [B,N,Hkv,D]
    (bf16); parent [B,N] int32; kv_len [B] int32 or None; out [B,N,Hq,D].
    k_tree = v_tree = None selects the tree-tail layout: node i's K/V are
    cache row kv_len[b] + i.
    """
    lib = load_library()
    B, N, Hq, D = q.shape
    Lmax, Hkv = k_cache.shape[1], k_cache.shape[2]
    dev = q.device
    _need(q, "q", torch.bfloat16, device=dev)
    _need(k_cache, "k_cache", torch.bfloat16, (B, Lmax, Hkv, D), dev)
    _need(v_cache, "v_cache", torch.bfloat16, (B, Lmax, Hkv, D), dev)
    _need_tree(k_tree, v_tree, (B, N, Hkv, D), dev)
    _need(parent, "parent", torch.int32, (B, N), dev)
    _need(out, "out", torch.bfloat16, (B, N, Hq, D), dev)
    if kv_len is not None:
        _need(kv_len, "kv_len", torch.int32, (B,), dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    need = lib.tv_tree_verify_attention_workspace(B, N, Hq, Hkv, D, Lmax)
    if need == 0:
        _check(-2)
    ws = workspace_tensor if workspace_tensor is not None else workspace("attn", need, dev, stream)
    _check(lib.tv_tree_verify_attention(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_tree), _ptr(v_tree), _ptr(parent),
        _ptr(kv_len), _ptr(out), B, N, Hq, Hkv, D, Lmax,
        0.0 if scale is None else float(scale), _ptr(ws), ws.numel(), ctypes.c_void_p(stream)))
    return out


def tree_verify_attention_paged(q, k_pool, v_pool, block_table, k_tree, v_tree, parent, out,
                                kv_len=None, scale=None, workspace_tensor=None):
    """tree_verify_attention over a paged cache: position t of sequence b is
    row t % block_size of k_pool/v_pool[block_table[b, t // block_size]].

    k_pool/v_pool [num_blocks, block_size, Hkv, D] bf16; block_table
    [B, max_blocks] int32; the rest as in tree_verify_attention.
    """
    lib = load_library()
    B, N, Hq, D = q.shape
    num_blocks, bs, Hkv = k_pool.shape[0], k_pool.shape[1], k_pool.shape[2]
    max_blocks = block_table.shape[1]
    dev = q.device
    _need(q, "q", torch.bfloat16, device=dev)
    _need(k_pool, "k_pool", torch.bfloat16, (num_blocks, bs, Hkv, D), dev)
    _need(v_pool, "v_pool", torch.bfloat16, (num_blocks, bs, Hkv, D), dev)
    _need(block_table, "block_table", torch.int32, (B, max_blocks), dev)
    _need_tree(k_tree, v_tree, (B, N, Hkv, D), dev)
    _need(parent, "parent", torch.int32, (B, N), dev)
    _need(out, "out", torch.bfloat16, (B, N, Hq, D), dev)
    if kv_len is not None:
        _need(kv_len, "kv_len", torch.int32, (B,), dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    need = lib.tv_tree_verify_attention_workspace(B, N, Hq, Hkv, D, max_blocks * bs)
    if need == 0:
        _check(-2)
    ws = workspace_tensor if workspace_tensor is not None else workspace("attn", need, dev, stream)
    _check(lib.tv_tree_verify_attention_paged(
        _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(block_table), bs, max_blocks, num_blocks,
        _ptr(k_tree), _ptr(v_tree), _ptr(parent), _ptr(kv_len), _ptr(out), B, N, Hq, Hkv, D,
        0.0 if scale is None else float(scale), _ptr(ws), ws.numel(), ctypes.c_void_p(stream)))
    return out


def block_causal_attention(q, k_ctx, v_ctx, k_blk, v_blk, anchors, out, scale=None,
                           workspace_tensor=None):
    """Attention under the draft head's training mask: position j of block k
    sees context rows < anchors[b, k] and positions 0..j of block k.

    q [B,A,S,Hq,D], k_ctx/v_ctx [B,L,Hkv,D], k_blk/v_blk [B,A,S,Hkv,D]
    (bf16); anchors [B,A] int32; out [B,A,S,Hq,D] bf16."""
    lib = load_library()
    B, A, S, Hq, D = q.shape
    L, Hkv = k_ctx.shape[1], k_ctx.shape[2]
    dev = q.device
    _need(q, "q", torch.bfloat16, device=dev)
    _need(k_ctx, "k_ctx", torch.bfloat16, (B, L, Hkv, D), dev)
    _need(v_ctx, "v_ctx", torch.bfloat16, (B, L, Hkv, D), dev)
    _need(k_blk, "k_blk", torch.bfloat16, (B, A, S, Hkv, D), dev)
    _need(v_blk, "v_blk", torch.bfloat16, (B, A, S, Hkv, D), dev)
    _need(anchors, "anchors", torch.int32, (B, A), dev)
    _need(out, "out", torch.bfloat16, (B, A, S, Hq, D), dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    need = lib.tv_block_causal_attention_workspace(B, A, S, Hq, Hkv, D, L)
    if need == 0:
        _check(-2)
    ws = workspace_tensor if workspace_tensor is not None else workspace("attn", need, dev, stream)
    _check(lib.tv_block_causal_attention(
        _ptr(q), _ptr(k_ctx), _ptr(v_ctx), _ptr(k_blk), _ptr(v_blk), _ptr(anchors), _ptr(out),
        B, A, S, Hq, Hkv, D, L, 0.0 if scale is None else float(scale), _ptr(ws), ws.numel(),
        ctypes.c_void_p(stream)))
    return out


def _dtype_code(t, name):
    if t.dtype == torch.bfloat16:
        return TV_BF16
    if t.dtype == torch.float32:
        return TV_F32
    raise ValueError(f"{name} must be bfloat16 or float32, got {t.dtype}")


def tree_accept_sampled(logits, draft_tok, parent, u_accept, seed, temperature, Dmax,
                        accept_len=None, path=None, correction=None, workspace_tensor=None):
    """Non-greedy tree acceptance (lossless multi-candidate rule for
    deterministic children).  logits [B,N,V] bf16 or fp32, draft_tok/parent
    [B,N] int32, u_accept [B,N] fp32.  Returns (accept_len [B], path
    [B,Dmax], correction [B]) int32."""
    lib = load_library()
    B, N, V = logits.shape
    dev = logits.device
    dt = _dtype_code(logits, "logits")
    _need(logits, "logits", logits.dtype, (B, N, V), dev)
    _need(draft_tok, "draft_tok", torch.int32, (B, N), dev)
    _need(parent, "parent", torch.int32, (B, N), dev)
    _need(u_accept, "u_accept", torch.float32, (B, N), dev)
    if accept_len is None:
        accept_len = torch.empty(B, dtype=torch.int32, device=dev)
    if path is None:
        path = torch.empty(B, Dmax, dtype=torch.int32, device=dev)
    if correction is None:
        correction = torch.empty(B, dtype=torch.int32, device=dev)
    _need(accept_len, "accept_len", torch.int32, (B,), dev)
    _need(path, "path", torch.int32, (B, Dmax), dev)
    _need(correction, "correction", torch.int32, (B,), dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    need = lib.tv_tree_accept_sampled_workspace(B, N, V)
    if need == 0:
        _check(-2)
    ws = workspace_tensor if workspace_tensor is not None else workspace("sample", need, dev,
                                                                         stream)
    _check(lib.tv_tree_accept_sampled(
        _ptr(logits), dt, _ptr(draft_tok), _ptr(parent), _ptr(u_accept),
        ctypes.c_ulonglong(int(seed) & 0xFFFFFFFFFFFFFFFF), ctypes.c_float(temperature), B, N, V,
        Dmax, _ptr(accept_len), _ptr(path), _ptr(correction), _ptr(ws), ws.numel(),
        ctypes.c_void_p(stream)))
    return accept_len, path, correction


def _tree_nodes(k_tree, n_nodes):
    if k_tree is not None:
        return k_tree.shape[1]
    if n_nodes is None:
        raise ValueError("the tree-tail layout (k_tree=None) needs n_nodes")
    return int(n_nodes)


def commit_path(k_tree, v_tree, path, accept_len, k_cache, v_cache, kv_len, n_nodes=None):
    """Append the accepted path's K/V (root first) to the contiguous cache at
    kv_len and advance kv_len, in place.  k_tree/v_tree [B,N,Hkv,D],
    path [B,Dmax], accept_len [B], k_cache/v_cache [B,Lmax,Hkv,D], kv_len [B].
    k_tree = v_tree = None: tree-tail layout (node i at cache row
    kv_len + i, N = n_nodes); the accepted rows are moved down in place."""
    lib = load_library()
    B, Lmax, Hkv, D = k_cache.shape
    N, Dmax = _tree_nodes(k_tree, n_nodes), path.shape[1]
    dev = k_cache.device
    _need_tree(k_tree, v_tree, (B, N, Hkv, D), dev)
    _need(path, "path", torch.int32, (B, Dmax), dev)
    _need(accept_len, "accept_len", torch.int32, (B,), dev)
    _need(k_cache, "k_cache", torch.bfloat16, (B, Lmax, Hkv, D), dev)
    _need(v_cache, "v_cache", torch.bfloat16, (B, Lmax, Hkv, D), dev)
    _need(kv_len, "kv_len", torch.int32, (B,), dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    _check(lib.tv_commit_path(
        _ptr(k_tree), _ptr(v_tree), _ptr(path), _ptr(accept_len), _ptr(k_cache), _ptr(v_cache),
        _ptr(kv_len), B, N, Hkv, D, Lmax, Dmax, ctypes.c_void_p(stream)))


def commit_path_paged(k_tree, v_tree, path, accept_len, k_pool, v_pool, block_table, kv_len,
                      n_nodes=None):
    """commit_path into a paged cache (layout as in
    tree_verify_attention_paged), in place; tree-tail layout as in
    commit_path."""
    lib = load_library()
    num_blocks, bs, Hkv, D = k_pool.shape
    B, max_blocks = block_table.shape
    N, Dmax = _tree_nodes(k_tree, n_nodes), path.shape[1]
    dev = k_pool.device
    _need_tree(k_tree, v_tree, (B, N, Hkv, D), dev)
    _need(path, "path", torch.int32, (B, Dmax), dev)
    _need(accept_len, "accept_len", torch.int32, (B,), dev)
    _need(k_pool, "k_pool", torch.bfloat16, (num_blocks, bs, Hkv, D), dev)
    _need(v_pool, "v_pool", torch.bfloat16, (num_blocks, bs, Hkv, D), dev)
    _need(block_table, "block_table", torch.int32, (B, max_blocks), dev)
    _need(kv_len, "kv_len", torch.int32, (B,), dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    _check(lib.tv_commit_path_paged(
        _ptr(k_tree), _ptr(v_tree), _ptr(path), _ptr(accept_len), _ptr(k_pool), _ptr(v_pool),
        _ptr(block_table), bs, max_blocks, num_blocks, _ptr(kv_len), B, N, Hkv, D, Dmax,
        ctypes.c_void_p(stream)))


def tree_accept(logits, draft_tok, parent, Dmax, accept_len=None, path=None,
                tgt_argmax=None, with_argmax=True, workspace_tensor=None):
    """Greedy tree acceptance.  Returns (accept_len [B], path [B,Dmax],
    tgt_argmax [B,N] or None), all int32 on the logits' device."""
    lib = load_library()
    B, N, V = logits.shape
    dev = logits.device
    if logits.dtype == torch.bfloat16:
        dt = TV_BF16
    elif logits.dtype == torch.float32:
        dt = TV_F32
    else:
        raise TypeError("logits must be bfloat16 or float32")
    _need(logits, "logits", logits.dtype, device=dev)
    _need(draft_tok, "draft_tok", torch.int32, (B, N), dev)
    _need(parent, "parent", torch.int32, (B, N), dev)
    if accept_len is None:
        accept_len = torch.empty(B, dtype=torch.int32, device=dev)
    if path is None:
        path = torch.empty(B, Dmax, dtype=torch.int32, device=dev)
    if tgt_argmax is None and with_argmax:
        tgt_argmax = torch.empty(B, N, dtype=torch.int32, device=dev)
    _need(accept_len, "accept_len", torch.int32, (B,), dev)
    _need(path, "path", torch.int32, (B, Dmax), dev)
    if tgt_argmax is not None:
        _need(tgt_argmax, "tgt_argmax", torch.int32, (B, N), dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    need = lib.tv_tree_accept_workspace(B, N, V)
    if need == 0:
        _check(-2)
    ws = workspace_tensor if workspace_tensor is not None else workspace("accept", need, dev, stream)
    _check(lib.tv_tree_accept(
        _ptr(logits), dt, _ptr(draft_tok), _ptr(parent), B, N, V, int(Dmax),
        _ptr(accept_len), _ptr(path), _ptr(tgt_argmax), _ptr(ws), ws.numel(),
        ctypes.c_void_p(stream)))
    return accept_len, path, tgt_argmax


def tree_accept_noalloc(logits, draft_tok, parent, Dmax, accept_len, path, tgt_argmax=None):
    """Greedy tree acceptance through the entry point that allocates nothing
    (its split keys live in the library's static per-GPU scratch).  The
    caller passes every output; returns (accept_len, path, tgt_argmax)."""
    lib = load_library()
    B, N, V = logits.shape
    dev = logits.device
    if logits.dtype == torch.bfloat16:
        dt = TV_BF16
    elif logits.dtype == torch.float32:
        dt = TV_F32
    else:
        raise TypeError("logits must be bfloat16 or float32")
    _need(logits, "logits", logits.dtype, device=dev)
    _need(draft_tok, "draft_tok", torch.int32, (B, N), dev)
    _need(parent, "parent", torch.int32, (B, N), dev)
    _need(accept_len, "accept_len", torch.int32, (B,), dev)
    _need(path, "path", torch.int32, (B, Dmax), dev)
    if tgt_argmax is not None:
        _need(tgt_argmax, "tgt_argmax", torch.int32, (B, N), dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    _check(lib.tv_tree_accept_noalloc(
        _ptr(logits), dt, _ptr(draft_tok), _ptr(parent), B, N, V, int(Dmax),
        _ptr(accept_len), _ptr(path), _ptr(tgt_argmax), ctypes.c_void_p(stream)))
    return accept_len, path, tgt_argmax


def draft_topw(logits, W, tok=None, logp=None, workspace_tensor=None):
    """(tok [B,Nd,W] int32, logp [B,Nd,W] fp32): the W largest draft logits
    of every draft depth and their log-probabilities.  logits [B,Nd,V]
    bfloat16 or float32."""
    lib = load_library()
    B, Nd, V = logits.shape
    dev = logits.device
    if logits.dtype == torch.bfloat16:
        dt = TV_BF16
    elif logits.dtype == torch.float32:
        dt = TV_F32
    else:
        raise TypeError("logits must be bfloat16 or float32")
    _need(logits, "logits", logits.dtype, device=dev)
    if tok is None:
        tok = torch.empty(B, Nd, W, dtype=torch.int32, device=dev)
    if logp is None:
        logp = torch.empty(B, Nd, W, dtype=torch.float32, device=dev)
    _need(tok, "tok", torch.int32, (B, Nd, W), dev)
    _need(logp, "logp", torch.float32, (B, Nd, W), dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    need = lib.tv_draft_topw_workspace(B, Nd, V)
    if need == 0:
        _check(-2)
    ws = workspace_tensor if workspace_tensor is not None else workspace("topw", need, dev, stream)
    _check(lib.tv_draft_topw(_ptr(logits), dt, B, Nd, V, int(W), _ptr(tok), _ptr(logp),
                             _ptr(ws), ws.numel(), ctypes.c_void_p(stream)))
    return tok, logp


def build_tree(tok, logp, budget, root_tok=None, with_score=True):
    """Best-first tree under a node budget from per-depth candidates
    (tok [B,Nd,W] int32, logp [B,Nd,W] fp32).  Returns (parent, token,
    depth, score or None, n_nodes); parent/token/depth are [B, budget]."""
    lib = load_library()
    B, Nd, W = tok.shape
    dev = tok.device
    _need(tok, "tok", torch.int32, (B, Nd, W), dev)
    _need(logp, "logp", torch.float32, (B, Nd, W), dev)
    if root_tok is not None:
        _need(root_tok, "root_tok", torch.int32, (B,), dev)
    parent = torch.empty(B, budget, dtype=torch.int32, device=dev)
    token = torch.empty(B, budget, dtype=torch.int32, device=dev)
    depth = torch.empty(B, budget, dtype=torch.int32, device=dev)
    score = torch.empty(B, budget, dtype=torch.float32, device=dev) if with_score else None
    n_nodes = torch.empty(B, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    _check(lib.tv_build_tree(_ptr(tok), _ptr(logp), _ptr(root_tok), B, Nd, W, int(budget),
                             _ptr(parent), _ptr(token), _ptr(depth), _ptr(score), _ptr(n_nodes),
                             ctypes.c_void_p(stream)))
    return parent, token, depth, score, n_nodes
