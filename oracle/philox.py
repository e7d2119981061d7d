"""Philox4x32-10 counter-based random numbers (test infrastructure only).

The generator of Salmon, Moraes, Dror and Shaw, "Parallel Random Numbers:
As Easy as 1, 2, 3" (SC 2011): a 4 x 32-bit counter is mixed with a
2 x 32-bit key by ten rounds of two 32x32 -> 64-bit multiplications, with
the key advanced by the Weyl increments between rounds.  Used where the
method draws more random numbers than can be passed in (one per vocabulary
entry for sampling a token), so that the GPU side and the oracle draw the
same numbers from the same definition.
"""
from __future__ import annotations

_M0, _M1 = 0xD2511F53, 0xCD9E8D57          # round multipliers
_W0, _W1 = 0x9E3779B9, 0xBB67AE85          # key increments (golden ratio, sqrt(3) - 1)
_MASK = 0xFFFFFFFF


def philox4x32(counter, key, rounds: int = 10):
    """Four 32-bit outputs for a 4-word counter and a 2-word key."""
    c0, c1, c2, c3 = (int(x) & _MASK for x in counter)
    k0, k1 = (int(x) & _MASK for x in key)
    for r in range(rounds):
        if r:
            k0 = (k0 + _W0) & _MASK
            k1 = (k1 + _W1) & _MASK
        p0 = _M0 * c0
        p1 = _M1 * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0, p1 & _MASK, (p0 >> 32) ^ c3 ^ k1, p0 & _MASK)
    return c0, c1, c2, c3


def uniform_open(word: int) -> float:
    """A 32-bit output as a number in (0, 1) from its top 23 bits:
    ((word >> 9) + 1/2) / 2^23.  Every value is exact in fp32 (the
    precision a GPU draws it in) and is never 0 or 1."""
    return ((int(word) >> 9) + 0.5) / 8388608.0


def philox4x32_array(c0, c1, c2, c3, k0: int, k1: int, rounds: int = 10):
    """philox4x32 over numpy arrays of counter words (one key); returns four
    uint64 arrays holding the 32-bit outputs."""
    import numpy as np
    m = np.uint64(_MASK)
    c0, c1, c2, c3 = (np.asarray(x, dtype=np.uint64) & m for x in (c0, c1, c2, c3))
    k0, k1 = int(k0) & _MASK, int(k1) & _MASK
    for r in range(rounds):
        if r:
            k0 = (k0 + _W0) & _MASK
            k1 = (k1 + _W1) & _MASK
        p0 = np.uint64(_M0) * c0
        p1 = np.uint64(_M1) * c2
        c0, c1, c2, c3 = ((p1 >> np.uint64(32)) ^ c1 ^ np.uint64(k0), p1 & m,
                          (p0 >> np.uint64(32)) ^ c3 ^ np.uint64(k1), p0 & m)
    return c0, c1, c2, c3
