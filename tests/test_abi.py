"""The C-ABI library loads, exports every symbol the header declares, and
rejects bad arguments on the host (no GPU needed: nothing is launched)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "treeverify.h")


def _lib():
    from paper_2606_18394_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        from paper_2606_18394_amd import build
        build.build()
    return binding.load_library()


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tv_\w+)\s*\(", src)))


def test_header_declares_the_api():
    names = _declared()
    for n in ["tv_tree_verify_attention", "tv_tree_accept", "tv_tree_verify_attention_workspace",
              "tv_tree_accept_workspace", "tv_status_string", "tv_version",
              "tv_draft_topw", "tv_draft_topw_workspace", "tv_build_tree",
              "tv_tree_verify_attention_paged", "tv_commit_path", "tv_commit_path_paged"]:
        assert n in names


def test_every_declared_symbol_is_exported():
    lib = _lib()
    for n in _declared():
        assert hasattr(lib, n), n


def test_status_strings_and_version():
    lib = _lib()
    assert lib.tv_version() == 2
    for code in [0, -1, -2, -3, -4, -5, -6, -7, -8]:
        assert lib.tv_status_string(code)
    assert b"unknown" in lib.tv_status_string(123)


def test_workspace_queries():
    lib = _lib()
    assert lib.tv_tree_verify_attention_workspace(1, 64, 32, 8, 128, 4096) > 0
    assert lib.tv_tree_verify_attention_workspace(1, 64, 30, 8, 128, 4096) == 0   # Hq % Hkv
    assert lib.tv_tree_verify_attention_workspace(1, 64, 32, 8, 96, 4096) == 0    # D
    assert lib.tv_tree_verify_attention_workspace(1, 4096, 32, 8, 128, 16) == 0   # N too big
    assert lib.tv_tree_verify_attention_workspace(0, 64, 32, 8, 128, 16) == 0
    assert lib.tv_tree_verify_attention_workspace(1, 16, 4, 2, 64, 0) > 0        # empty cache ok
    assert lib.tv_tree_accept_workspace(1, 64, 151936) > 0
    assert lib.tv_tree_accept_workspace(1, 0, 10) == 0
    assert lib.tv_tree_accept_workspace(1, 4096, 10) == 0
    assert lib.tv_draft_topw_workspace(1, 8, 151936) > 0
    assert lib.tv_draft_topw_workspace(1, 65, 10) == 0     # draft depth above the limit
    assert lib.tv_draft_topw_workspace(1, 8, 0) == 0


FAKE = 0x100000  # 16-byte aligned non-null address; never dereferenced


def _attn(lib, **kw):
    a = dict(q=FAKE, kc=FAKE, vc=FAKE, kt=FAKE, vt=FAKE, parent=FAKE, kv_len=None, out=FAKE,
             B=1, N=64, Hq=32, Hkv=8, D=128, Lmax=4096, scale=0.0, ws=FAKE, wsb=1 << 40)
    a.update(kw)
    return lib.tv_tree_verify_attention(
        a["q"], a["kc"], a["vc"], a["kt"], a["vt"], a["parent"], a["kv_len"], a["out"],
        a["B"], a["N"], a["Hq"], a["Hkv"], a["D"], a["Lmax"], ctypes.c_float(a["scale"]),
        a["ws"], a["wsb"], None)


def _acc(lib, **kw):
    a = dict(logits=FAKE, dt=0, draft=FAKE, parent=FAKE, B=1, N=64, V=151936, Dmax=9,
             ln=FAKE, path=FAKE, tgt=None, ws=FAKE, wsb=1 << 40)
    a.update(kw)
    return lib.tv_tree_accept(a["logits"], a["dt"], a["draft"], a["parent"], a["B"], a["N"],
                              a["V"], a["Dmax"], a["ln"], a["path"], a["tgt"], a["ws"],
                              a["wsb"], None)


def test_attention_host_errors():
    lib = _lib()
    assert _attn(lib, q=None) == -1
    assert _attn(lib, out=None) == -1
    assert _attn(lib, parent=None) == -1
    assert _attn(lib, kc=None) == -1
    assert _attn(lib, B=0) == -2
    assert _attn(lib, N=0) == -2
    assert _attn(lib, Hq=30) == -2
    assert _attn(lib, Lmax=-1) == -2
    assert _attn(lib, D=96) == -4
    assert _attn(lib, N=2049) == -4
    assert _attn(lib, q=FAKE + 8) == -7
    assert _attn(lib, out=FAKE + 2) == -7
    assert _attn(lib, ws=None) == -5
    assert _attn(lib, wsb=16) == -5


def test_accept_host_errors():
    lib = _lib()
    assert _acc(lib, logits=None) == -1
    assert _acc(lib, path=None) == -1
    assert _acc(lib, ln=None) == -1
    assert _acc(lib, dt=7) == -3
    assert _acc(lib, B=0) == -2
    assert _acc(lib, V=0) == -2
    assert _acc(lib, Dmax=0) == -2
    assert _acc(lib, N=2049) == -4
    assert _acc(lib, ws=None) == -5
    assert _acc(lib, wsb=8) == -5
    assert _acc(lib, ws=FAKE + 4) == -7


def test_accept_noalloc_host_errors():
    """The allocation-free acceptance checks its sizes before it touches a
    GPU: errors come back with nothing launched."""
    lib = _lib()

    def call(**kw):
        a = dict(logits=FAKE, dt=0, draft=FAKE, parent=FAKE, B=1, N=64, V=151936, Dmax=9,
                 ln=FAKE, path=FAKE, tgt=None)
        a.update(kw)
        return lib.tv_tree_accept_noalloc(a["logits"], a["dt"], a["draft"], a["parent"], a["B"],
                                          a["N"], a["V"], a["Dmax"], a["ln"], a["path"],
                                          a["tgt"], None)
    assert call(logits=None) == -1
    assert call(path=None) == -1
    assert call(dt=3) == -3
    assert call(B=0) == -2
    assert call(N=2049) == -4
    # split keys beyond the static scratch: 1.2M node rows
    assert lib.tv_tree_accept_workspace(600, 2048, 8) > (8 << 20)
    assert call(B=600, N=2048, V=8) == -8
    assert b"TV_ERR_SCRATCH" in lib.tv_status_string(-8)


def test_binding_refuses_cpu_tensors():
    import torch
    from paper_2606_18394_amd import tree_accept
    _lib()
    with pytest.raises(ValueError):
        tree_accept(torch.zeros(1, 2, 8), torch.zeros(1, 2, dtype=torch.int32),
                    torch.tensor([[-1, 0]], dtype=torch.int32), 2)


def _topw(lib, **kw):
    a = dict(logits=FAKE, dt=0, B=1, Nd=8, V=151936, W=4, tok=FAKE, logp=FAKE, ws=FAKE,
             wsb=1 << 40)
    a.update(kw)
    return lib.tv_draft_topw(a["logits"], a["dt"], a["B"], a["Nd"], a["V"], a["W"], a["tok"],
                             a["logp"], a["ws"], a["wsb"], None)


def _build(lib, **kw):
    a = dict(tok=FAKE, logp=FAKE, root=None, B=1, Nd=8, W=4, budget=64, parent=FAKE,
             token=FAKE, depth=FAKE, score=None, n=FAKE)
    a.update(kw)
    return lib.tv_build_tree(a["tok"], a["logp"], a["root"], a["B"], a["Nd"], a["W"],
                             a["budget"], a["parent"], a["token"], a["depth"], a["score"],
                             a["n"], None)


def test_drafting_host_errors():
    lib = _lib()
    assert _topw(lib, logits=None) == -1
    assert _topw(lib, logp=None) == -1
    assert _topw(lib, dt=5) == -3
    assert _topw(lib, W=0) == -2
    assert _topw(lib, V=3, W=4) == -2          # fewer tokens than candidates
    assert _topw(lib, W=17) == -4
    assert _topw(lib, Nd=65) == -4
    assert _topw(lib, ws=None) == -5
    assert _topw(lib, wsb=8) == -5
    assert _topw(lib, ws=FAKE + 4) == -7
    assert _build(lib, tok=None) == -1
    assert _build(lib, n=None) == -1
    assert _build(lib, budget=0) == -2
    assert _build(lib, B=0) == -2
    assert _build(lib, budget=2049) == -4
    assert _build(lib, W=17) == -4
    assert _build(lib, Nd=65) == -4


def _attn_paged(lib, **kw):
    a = dict(q=FAKE, kp=FAKE, vp=FAKE, bt=FAKE, bs=256, mb=16, nb=64, kt=FAKE, vt=FAKE,
             parent=FAKE, kv_len=None, out=FAKE, B=1, N=64, Hq=32, Hkv=8, D=128, scale=0.0,
             ws=FAKE, wsb=1 << 40)
    a.update(kw)
    return lib.tv_tree_verify_attention_paged(
        a["q"], a["kp"], a["vp"], a["bt"], a["bs"], a["mb"], a["nb"], a["kt"], a["vt"],
        a["parent"], a["kv_len"], a["out"], a["B"], a["N"], a["Hq"], a["Hkv"], a["D"],
        ctypes.c_float(a["scale"]), a["ws"], a["wsb"], None)


def test_paged_attention_host_errors():
    lib = _lib()
    assert _attn_paged(lib, bs=48) == -2          # not a power of two
    assert _attn_paged(lib, bs=16) == -2          # below the smallest block
    assert _attn_paged(lib, mb=-1) == -2
    assert _attn_paged(lib, nb=-1) == -2
    assert _attn_paged(lib, bt=None) == -1
    assert _attn_paged(lib, nb=0) == -1           # a cache but no pool
    assert _attn_paged(lib, kp=None) == -1
    assert _attn_paged(lib, q=None) == -1
    assert _attn_paged(lib, Hq=30) == -2
    assert _attn_paged(lib, D=96) == -4
    assert _attn_paged(lib, kp=FAKE + 8) == -7
    assert _attn_paged(lib, ws=None) == -5
    assert _attn_paged(lib, mb=1 << 20, bs=1 << 11) == -4   # capacity above 2^30


def _commit(lib, **kw):
    a = dict(kt=FAKE, vt=FAKE, path=FAKE, ln=FAKE, kc=FAKE, vc=FAKE, kvl=FAKE, B=1, N=64,
             Hkv=8, D=128, Lmax=4096, Dmax=9)
    a.update(kw)
    return lib.tv_commit_path(a["kt"], a["vt"], a["path"], a["ln"], a["kc"], a["vc"], a["kvl"],
                              a["B"], a["N"], a["Hkv"], a["D"], a["Lmax"], a["Dmax"], None)


def _commit_paged(lib, **kw):
    a = dict(kt=FAKE, vt=FAKE, path=FAKE, ln=FAKE, kp=FAKE, vp=FAKE, bt=FAKE, bs=256, mb=16,
             nb=64, kvl=FAKE, B=1, N=64, Hkv=8, D=128, Dmax=9)
    a.update(kw)
    return lib.tv_commit_path_paged(a["kt"], a["vt"], a["path"], a["ln"], a["kp"], a["vp"],
                                    a["bt"], a["bs"], a["mb"], a["nb"], a["kvl"], a["B"],
                                    a["N"], a["Hkv"], a["D"], a["Dmax"], None)


def test_commit_host_errors():
    lib = _lib()
    assert _commit(lib, kt=None) == -1
    assert _commit(lib, path=None) == -1
    assert _commit(lib, kvl=None) == -1
    assert _commit(lib, B=0) == -2
    assert _commit(lib, Lmax=0) == -2
    assert _commit(lib, Dmax=0) == -2
    assert _commit(lib, D=96) == -4
    assert _commit(lib, N=2049) == -4
    assert _commit(lib, kc=FAKE + 8) == -7
    assert _commit_paged(lib, bt=None) == -1
    assert _commit_paged(lib, bs=100) == -2
    assert _commit_paged(lib, mb=0) == -2
    assert _commit_paged(lib, nb=0) == -2
    assert _commit_paged(lib, vp=FAKE + 2) == -7
    assert _commit_paged(lib, D=80) == -4


def test_tree_tail_host_errors():
    lib = _lib()
    assert _attn(lib, kt=None) == -1                         # only one of the two NULL
    assert _attn(lib, vt=None) == -1
    assert _attn(lib, kt=None, vt=None, N=64, Lmax=63) == -2  # no room for the tree
    assert _attn(lib, kt=None, vt=None, N=64, Lmax=0) == -2
    assert _attn_paged(lib, kt=None) == -1
    assert _attn_paged(lib, kt=None, vt=None, N=64, mb=1, bs=32) == -2
    assert _commit(lib, vt=None) == -1
    assert _commit(lib, kt=None, vt=None, N=64, Lmax=63) == -2
    assert _commit_paged(lib, kt=None, vt=None, N=64, mb=1, bs=32) == -2


def _bc(lib, **kw):
    a = dict(q=FAKE, kc=FAKE, vc=FAKE, kb=FAKE, vb=FAKE, anc=FAKE, out=FAKE, B=1, A=512, S=16,
             Hq=32, Hkv=8, D=128, L=4096, scale=0.0, ws=FAKE, wsb=1 << 40)
    a.update(kw)
    return lib.tv_block_causal_attention(
        a["q"], a["kc"], a["vc"], a["kb"], a["vb"], a["anc"], a["out"], a["B"], a["A"], a["S"],
        a["Hq"], a["Hkv"], a["D"], a["L"], ctypes.c_float(a["scale"]), a["ws"], a["wsb"], None)


def test_block_causal_host_errors():
    lib = _lib()
    assert lib.tv_block_causal_attention_workspace(1, 512, 16, 32, 8, 128, 4096) > 0
    assert lib.tv_block_causal_attention_workspace(1, 0, 16, 32, 8, 128, 4096) == 0
    assert lib.tv_block_causal_attention_workspace(1, 4, 2049, 32, 8, 128, 64) == 0
    assert _bc(lib, anc=None) == -1
    assert _bc(lib, kb=None) == -1
    assert _bc(lib, kc=None) == -1
    assert _bc(lib, A=0) == -2
    assert _bc(lib, S=0) == -2
    assert _bc(lib, Hq=30) == -2
    assert _bc(lib, D=80) == -4
    assert _bc(lib, S=2049) == -4
    assert _bc(lib, B=1 << 13, A=1 << 12) == -4
    assert _bc(lib, out=FAKE + 4) == -7
    assert lib.tv_block_causal_attention_workspace(1, 4, 16, 32, 8, 128, 4096) > 256  # splits
    assert _bc(lib, A=4, ws=None) == -5


def _samp(lib, **kw):
    a = dict(lg=FAKE, dt=0, tok=FAKE, par=FAKE, u=FAKE, seed=1, T=1.0, B=1, N=64,
             V=151936, Dmax=9, ln=FAKE, path=FAKE, corr=FAKE, ws=FAKE, wsb=1 << 40)
    a.update(kw)
    return lib.tv_tree_accept_sampled(
        a["lg"], a["dt"], a["tok"], a["par"], a["u"], a["seed"], ctypes.c_float(a["T"]),
        a["B"], a["N"], a["V"], a["Dmax"], a["ln"], a["path"], a["corr"], a["ws"], a["wsb"],
        None)


def test_sampled_accept_host_errors():
    lib = _lib()
    assert lib.tv_tree_accept_sampled_workspace(1, 64, 151936) > 0
    assert lib.tv_tree_accept_sampled_workspace(1, 64, 1 << 23) > 0
    assert lib.tv_tree_accept_sampled_workspace(1, 64, (1 << 23) + 1) == 0
    assert lib.tv_tree_accept_sampled_workspace(1, 0, 100) == 0
    assert _samp(lib, lg=None) == -1
    assert _samp(lib, u=None) == -1
    assert _samp(lib, corr=None) == -1
    assert _samp(lib, dt=2) == -3
    assert _samp(lib, T=0.0) == -2
    assert _samp(lib, T=-1.0) == -2
    assert _samp(lib, T=float("inf")) == -2
    assert _samp(lib, T=float("nan")) == -2
    assert _samp(lib, V=(1 << 23) + 8) == -4
    assert _samp(lib, N=2049) == -4
    assert _samp(lib, Dmax=0) == -2
    assert _samp(lib, ws=None) == -5
    assert _samp(lib, wsb=64) == -5
    assert _samp(lib, ws=FAKE + 8) == -7


def test_plain_c_program_compiles_against_the_header(tmp_path):
    """The header is plain C99 and the library links from C (the program
    itself runs in the GPU suite)."""
    from paper_2606_18394_amd import build
    if not os.path.exists(build.LIB):
        build.build()
    exe = build.build_example(out=str(tmp_path / "abi_example"))
    assert os.path.exists(exe)
