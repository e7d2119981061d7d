"""Launch-plan invariants checked on the host: the plan header is plain C++,
compiled here with g++, and every workgroup's decoded work item is checked
for range, uniqueness and workspace/LDS bounds."""
import os
import shutil
import subprocess

import pytest

from paper_2606_18394_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_18394_amd", "csrc")


def shapes():
    out = []
    for name in synth.WORKLOAD_ORDER:
        w = synth.WORKLOADS[name]
        out.append((w.B, w.N, w.Hq, w.Hkv, w.D, w.L, w.V))
    for B in [1, 3, 16]:
        for N in [1, 2, 17, 64, 65, 129, 512, 2048]:
            for Hq, Hkv in [(4, 4), (8, 2), (32, 8), (64, 8), (24, 8), (2, 1)]:
                for D in [64, 128]:
                    for L in [0, 1, 64, 1000, 32768]:
                        out.append((B, N, Hq, Hkv, D, L, 151936 if N < 100 else 1001))
    # more row blocks than the split-KV sync region holds: no split
    out += [(64, 512, 64, 8, 128, 1000, 1001), (512, 64, 32, 8, 128, 32768, 1001)]
    return out


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_plans(tmp_path):
    exe = tmp_path / "plan_check"
    subprocess.run(["g++", "-O1", "-std=c++17", "-I", CSRC,
                    os.path.join(ROOT, "tests", "native", "plan_check.cpp"), "-o", str(exe)],
                   check=True)
    data = "\n".join(" ".join(map(str, s)) for s in shapes()) + "\n"
    res = subprocess.run([str(exe)], input=data, capture_output=True, text=True)
    fails = [l for l in res.stdout.splitlines() if l.startswith("FAIL")]
    assert res.returncode == 0 and not fails, "\n".join(fails[:20]) + res.stdout[-300:]


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_plans_under_host_sanitizers(tmp_path):
    """The same checks with AddressSanitizer and UndefinedBehaviorSanitizer on
    the host planner (integer overflow in sizes, out-of-range indexing)."""
    exe = tmp_path / "plan_check_san"
    build = subprocess.run(["g++", "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined",
                            "-fno-sanitize-recover=undefined", "-I", CSRC,
                            os.path.join(ROOT, "tests", "native", "plan_check.cpp"), "-o", str(exe)],
                           capture_output=True, text=True)
    if build.returncode != 0:
        pytest.skip("host sanitizer runtime not available: " + build.stderr[-200:])
    data = "\n".join(" ".join(map(str, s)) for s in shapes()) + "\n"
    res = subprocess.run([str(exe)], input=data, capture_output=True, text=True)
    fails = [l for l in res.stdout.splitlines() if l.startswith("FAIL")]
    assert res.returncode == 0 and not fails, "\n".join(fails[:20]) + res.stderr[-1000:]


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_accept_split_rule(tmp_path):
    """The acceptance scan's split count: the ~2048-workgroup target (at most
    16 splits, at least one full round of loads each), then down to half of
    it the count whose load slots are best used.  Checked against a plain
    re-derivation of that rule, and at the measured shapes: 512 rows of
    151936 bf16 logits take 2 splits (4 leave 23% of the slots empty), 128
    and 64 rows keep 10."""
    exe = tmp_path / "accept_split_check"
    subprocess.run(["g++", "-O1", "-std=c++17", "-I", CSRC,
                    os.path.join(ROOT, "tests", "native", "accept_split_check.cpp"), "-o", str(exe)],
                   check=True)
    cases = [(1, 512, 151936, 2), (1, 128, 151936, 2), (1, 64, 151936, 2), (16, 64, 151936, 2),
             (1, 16, 1024, 4), (3, 100, 50000, 2), (1, 2048, 151936, 4), (7, 33, 32000, 4)]
    res = subprocess.run([str(exe)], input="".join(f"{b} {n} {v} {e}\n" for b, n, v, e in cases),
                         capture_output=True, text=True, check=True)
    got = {tuple(map(int, l.split()[:4])): int(l.split()[4]) for l in res.stdout.splitlines()}

    def rule(b, n, v, esize):
        rows, per_round = b * n, 512 * 4
        chunks = -(-v // (16 // esize))
        ns = min(16, max(1, -(-2048 // rows)), -(-chunks // per_round))
        ns = max(ns, 1)

        def fill(k):
            c = -(-chunks // k)
            return c / (-(-c // per_round) * per_round)
        best = ns
        for k in range(ns - 1, 0, -1):
            if 2 * k < ns:
                break
            if fill(k) > fill(best) + 1e-9:
                best = k
        return best
    for c in cases:
        assert got[c] == rule(*c), (c, got[c], rule(*c))
    assert got[(1, 512, 151936, 2)] == 2
    assert got[(1, 128, 151936, 2)] == 10 and got[(1, 64, 151936, 2)] == 10
