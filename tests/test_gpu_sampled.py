"""GPU parity of non-greedy tree acceptance (Sec. 2.4 speculative sampling
along tree branches) against the oracle, through the C ABI.

The acceptance tests and the race are decided in fp32 on the GPU and in
fp64 in the oracle.  Inputs are drawn so that no node's test lies within
1e-4 (relative) of its threshold, which makes path and accept_len unique
and bit-exact; a correction token whose race is within 1e-3 of a tie may
be either of the two leaders."""
import numpy as np
import pytest
import torch

import oracle
from oracle.tree_accept_sampled import tree_accept_sampled as oracle_sampled
from paper_2606_18394_amd import synth
from helpers import dev_bf16, dev_i32

pytestmark = pytest.mark.gpu

CASES = [
    # (B, N, V, Nd, depth cap, T, dtype target, dtype draft, p_match)
    (3, 20, 1000, 5, 5, 1.0, "bf16", "bf16", 0.5),
    (2, 33, 999, 6, 6, 1.0, "f32", "bf16", 0.5),
    (4, 17, 4096, 4, 4, 0.6, "bf16", "f32", 0.3),
    (1, 64, 151936, 8, 8, 1.0, "bf16", "bf16", 0.6),
    (16, 64, 151936, 8, 8, 1.0, "bf16", "bf16", 0.5),
    (2, 300, 2048, 12, 12, 1.3, "f32", "f32", 0.7),
    (1, 1, 64, 1, 1, 1.0, "bf16", "bf16", 0.5),
]


def _logits(rng, shape, dtype, std=2.0):
    x = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(std)
    if dtype == "f32":
        return x, torch.from_numpy(x).cuda(), x.astype(np.float64)
    bits = synth.bf16_bits(x)
    return bits, dev_bf16(bits), oracle.decode_bf16(bits)


def _inputs(case):
    B, N, V, Nd, depth, T, dt, ddt, pm = CASES[case]
    rng = np.random.default_rng(2000 + case)
    par = np.stack([synth.random_tree(rng, N, depth=min(depth, max(N - 1, 1)), branching=4)
                    if N > 1 else np.array([-1], np.int32) for _ in range(B)])
    _, lg_d, lg64 = _logits(rng, (B, N, V), dt)
    _, dl_d, dl64 = _logits(rng, (B, Nd, V), ddt)
    # draft tokens: the target's most likely token at the parent with
    # probability p_match, else uniform
    tok = rng.integers(0, V, size=(B, N)).astype(np.int32)
    best = lg64.argmax(-1)
    for b in range(B):
        for i in range(1, N):
            if rng.random() < pm:
                tok[b, i] = best[b, par[b, i]]
    seed = int(rng.integers(0, 2**63))
    u = rng.random((B, N), dtype=np.float32)
    for _ in range(20):   # keep every test clear of its threshold
        res = oracle_sampled(lg64, dl64, tok, par, u.astype(np.float64), seed, T, depth + 1,
                             detail=True)
        close = res[3]["margin"] < 1e-4
        if not close.any():
            break
        u[close] = rng.random(int(close.sum()), dtype=np.float32)
    assert not close.any()
    return dict(par=par, tok=tok, u=u, seed=seed, T=T, Dmax=depth + 1, lg_d=lg_d, dl_d=dl_d,
                ref=res)


def _gpu(x):
    from paper_2606_18394_amd import tree_accept_sampled
    ln, path, corr = tree_accept_sampled(x["lg_d"], x["dl_d"], dev_i32(x["tok"]),
                                         dev_i32(x["par"]), torch.from_numpy(x["u"]).cuda(),
                                         x["seed"], x["T"], x["Dmax"])
    torch.cuda.synchronize()
    return ln.cpu().numpy(), path.cpu().numpy(), corr.cpu().numpy()


def _check(got, ref):
    ln, path, corr = got
    eln, epath, ecorr, det = ref
    np.testing.assert_array_equal(ln, eln)
    np.testing.assert_array_equal(path, epath)
    for b in range(len(ln)):
        if det["gap"][b] < 1e-3:
            assert corr[b] in (ecorr[b], det["runner_up"][b]), b
        else:
            assert corr[b] == ecorr[b], (b, corr[b], ecorr[b])


@pytest.mark.parametrize("case", range(len(CASES)))
def test_sampled_parity(case):
    print(f"sampled case {CASES[case]}", flush=True)
    x = _inputs(case)
    got = _gpu(x)
    print(f"accept_len {got[0][:8].tolist()} correction {got[2][:8].tolist()}")
    _check(got, x["ref"])


def test_sampled_invalid_and_too_deep():
    x = _inputs(0)
    par = x["par"].copy()
    par[0, 5] = 7                 # parent after child
    x["par"] = par
    got = _gpu(x)
    assert got[0][0] == -1 and got[2][0] == -1 and (got[1][0] == -1).all()
    # trees deeper than the draft logits reach
    y = _inputs(2)
    y["dl_d"] = y["dl_d"][:, :2].contiguous()
    got = _gpu(y)
    ref = oracle_sampled(
        *(t.float().cpu().numpy().astype(np.float64) for t in (y["lg_d"], y["dl_d"])),
        y["tok"], y["par"], y["u"].astype(np.float64), y["seed"], y["T"], y["Dmax"])
    np.testing.assert_array_equal(got[0], ref[0])
    np.testing.assert_array_equal(got[2], ref[2])


def test_sampled_equal_distributions_accept_the_chain():
    """Draft logits equal to the target's at the parent: every ratio is 1,
    the whole chain is accepted and the correction is drawn from p at the
    leaf."""
    from paper_2606_18394_amd import tree_accept_sampled
    rng = np.random.default_rng(7)
    N, V = 9, 512
    lg = rng.standard_normal((1, N, V), dtype=np.float32)
    dl = lg[:, :N - 1].copy()
    par = np.arange(-1, N - 1, dtype=np.int32)[None]
    tok = rng.integers(0, V, size=(1, N)).astype(np.int32)
    u = np.full((1, N), 0.5, np.float32)
    ln, path, corr = tree_accept_sampled(torch.from_numpy(lg).cuda(), torch.from_numpy(dl).cuda(),
                                         dev_i32(tok), dev_i32(par), torch.from_numpy(u).cuda(),
                                         123, 1.0, N)
    torch.cuda.synchronize()
    eln, epath, ecorr = oracle_sampled(lg.astype(np.float64), dl.astype(np.float64), tok, par,
                                       u.astype(np.float64), 123, 1.0, N)
    assert ln.item() == N == eln[0]
    assert path.cpu().numpy()[0].tolist() == list(range(N))
    assert corr.item() == ecorr[0]
