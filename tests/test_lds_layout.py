"""Bank model of the attention kernel's LDS tile layout (host only).

The tile layout XOR-swizzles the 16-byte chunks of every key row (the
TileLayout rule in tv_attention.hip, restated here).  This models the two
operand reads of a tile -- the K reads (ds_read_b128, lane (g4, l16) reads
row 16 tt + l16 at chunk 4 cc + g4) and the transposing V reads
(ds_read_b64_tr_b16, lane (g4, l16) reads row 4 g4 + l16 / 4 (+16), chunk
2 dt + (l16 % 4) / 2, half l16 % 2) -- under two ways of serving a read: 256
bytes per cycle (64 banks of 4 bytes) and 128 bytes per cycle (32 banks).
The committed rule is conflict-free at 64 banks and 2-way on the K reads at
32 banks: one cycle in three of the reads is a conflict cycle, the ratio the
hardware counters report for the kernel (SQ_LDS_BANK_CONFLICT over
SQ_LDS_IDX_ACTIVE = 8.68 M / 26.1 M at the largest tree)."""
import pytest


def swz_committed(D, r):
    return (((r & 7) << 1) | ((r >> 3) & 1)) if D == 128 else \
        ((((r >> 1) & 3) << 1) | ((r >> 3) & 1))


def swz_both(D, r):
    """Conflict-free at both widths (measured no faster, not used)."""
    hi = ((r >> 2) ^ (r >> 3)) & 1
    return (((r & 3) << 1) | ((r >> 2) & 1) | (hi << 3)) if D == 128 else \
        ((((r & 3) ^ ((r >> 2) & 1)) << 1) ^ hi)


def _off(D, swz, r, ch):
    return r * 2 * D + ((ch ^ swz(D, r)) << 4)


def _reads(D, swz):
    k = [(16, [_off(D, swz, 16 * tt + (l & 15), 4 * cc + (l >> 4)) for l in range(64)])
         for tt in range(2) for cc in range(D // 32)]
    v = []
    for dt in range(D // 16):
        for hi in range(2):
            v.append((8, [_off(D, swz, 4 * (l >> 4) + ((l & 15) >> 2) + 16 * hi,
                               2 * dt + (((l & 15) & 3) >> 1)) + 8 * (l & 1) for l in range(64)]))
    return k, v


def _cycles(reads, banks):
    """Cycles of a list of (bytes per lane, addresses): each pass serves
    banks * 4 bytes of lanes; a pass takes as many cycles as the most
    distinct words any one bank must deliver."""
    total = 0
    for size, addrs in reads:
        lanes = banks * 4 // size
        for p0 in range(0, 64, lanes):
            use = {}
            for a in addrs[p0:p0 + lanes]:
                for w in range(size // 4):
                    use.setdefault((a // 4 + w) % banks, set()).add(a // 4 + w)
            total += max(len(s) for s in use.values())
    return total


def _ideal(reads, banks):
    return sum(64 * size // (banks * 4) for size, _ in reads)


@pytest.mark.parametrize("D", [64, 128])
def test_swizzle_is_a_permutation_of_each_row(D):
    for swz in (swz_committed, swz_both):
        for r in range(32):
            assert sorted(c ^ swz(D, r) for c in range(D // 8)) == list(range(D // 8))


@pytest.mark.parametrize("D", [64, 128])
def test_committed_rule_is_conflict_free_at_64_banks(D):
    k, v = _reads(D, swz_committed)
    assert _cycles(k, 64) == _ideal(k, 64) and _cycles(v, 64) == _ideal(v, 64)


def test_committed_rule_at_32_banks_matches_the_counters():
    k, v = _reads(128, swz_committed)
    assert _cycles(v, 32) == _ideal(v, 32)          # V reads stay conflict-free
    assert _cycles(k, 32) == 2 * _ideal(k, 32)      # K reads are 2-way
    total = _cycles(k, 32) + _cycles(v, 32)
    extra = total - _ideal(k, 32) - _ideal(v, 32)
    assert abs(extra / total - 8.677e6 / 26.128e6) < 0.01


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("banks", [32, 64])
def test_alternative_rule_is_conflict_free_at_both_widths(D, banks):
    k, v = _reads(D, swz_both)
    assert _cycles(k, banks) == _ideal(k, banks) and _cycles(v, banks) == _ideal(v, banks)
