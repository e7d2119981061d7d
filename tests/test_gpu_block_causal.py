"""GPU parity of attention under the draft head's training mask (App.
Training Details) against the fp64 oracle, through the C ABI.  Bar: max-abs
error <= 1e-2 on bf16 N(0,1) inputs."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_18394_amd import synth
from helpers import dev_bf16, dev_i32

pytestmark = pytest.mark.gpu
TOL = 1e-2

CASES = [
    # (B, A, S, Hq, Hkv, D, L, anchors: "rand" | list per example)
    (1, 4, 16, 32, 8, 128, 512, [[0, 511, 512, 100]]),
    (2, 3, 5, 8, 2, 64, 97, [[-4, 50, 200], [1, 31, 33]]),
    (1, 2, 1, 4, 4, 128, 64, [[0, 64]]),
    (3, 7, 16, 16, 2, 128, 300, "rand"),
    (1, 1, 16, 8, 8, 64, 0, [[0]]),
    (2, 64, 16, 32, 8, 128, 1024, "rand"),
    (1, 512, 16, 32, 8, 128, 4096, "rand"),
]


def _inputs(case):
    B, A, S, Hq, Hkv, D, L, anc = CASES[case]
    rng = np.random.default_rng(1500 + case)
    anchors = (rng.integers(0, L + 1, size=(B, A)) if anc == "rand" else np.array(anc))
    return dict(
        anchors=anchors.astype(np.int32),
        q=synth._normal_bf16(rng, (B, A, S, Hq, D)),
        k_ctx=synth._normal_bf16(rng, (B, L, Hkv, D)),
        v_ctx=synth._normal_bf16(rng, (B, L, Hkv, D)),
        k_blk=synth._normal_bf16(rng, (B, A, S, Hkv, D)),
        v_blk=synth._normal_bf16(rng, (B, A, S, Hkv, D)))


@pytest.mark.parametrize("case", range(len(CASES)))
def test_block_causal_parity(case):
    from paper_2606_18394_amd import block_causal_attention
    B, A, S, Hq, Hkv, D, L, _ = CASES[case]
    print(f"block-causal case {CASES[case][:7]}", flush=True)
    x = _inputs(case)
    out = torch.full((B, A, S, Hq, D), 7.0, dtype=torch.bfloat16, device="cuda")
    block_causal_attention(dev_bf16(x["q"]), dev_bf16(x["k_ctx"]), dev_bf16(x["v_ctx"]),
                           dev_bf16(x["k_blk"]), dev_bf16(x["v_blk"]), dev_i32(x["anchors"]),
                           out)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    assert np.isfinite(got).all()
    dec = oracle.decode_bf16
    # Every block is checked.  Blocks see nothing of each other (an oracle
    # invariant pinned on the CPU), so the oracle runs on groups of at most
    # 16 blocks at a time, which bounds the dense mask it builds.
    err = 0.0
    grp = 16
    for b in range(B):
        for k0 in range(0, A, grp):
            ks = slice(k0, min(A, k0 + grp))
            ref = oracle.block_causal_attention(
                dec(x["q"][b:b + 1, ks]), dec(x["k_ctx"][b:b + 1]), dec(x["v_ctx"][b:b + 1]),
                dec(x["k_blk"][b:b + 1, ks]), dec(x["v_blk"][b:b + 1, ks]),
                x["anchors"][b:b + 1, ks])
            err = max(err, float(np.abs(got[b:b + 1, ks] - ref).max()))
    print(f"max abs err {err:.3e} over all {B * A} blocks", flush=True)
    assert err <= TOL
