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
