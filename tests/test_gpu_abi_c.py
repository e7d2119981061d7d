"""The C ABI driven from a plain C program (tests/native/abi_example.c), with
device buffers from the HIP runtime and no Python on the call path."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "native", "abi_example.c")
EXE = os.path.join(ROOT, "tests", "native", "abi_example")

pytestmark = pytest.mark.gpu


def _exe():
    from paper_2606_18394_amd import build
    if not os.path.exists(build.LIB):
        build.build()
    if not os.path.exists(EXE) or os.path.getmtime(EXE) < os.path.getmtime(SRC):
        build.build_example()
    return EXE


def test_c_program_runs_a_verification_step():
    exe = _exe()
    env = dict(os.environ)
    env["LD_LIBRARY_PATH"] = os.path.dirname(os.path.abspath(
        os.path.join(ROOT, "paper_2606_18394_amd", "libtreeverify.so"))) + ":" + \
        env.get("LD_LIBRARY_PATH", "")
    print("running", exe, flush=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=env)
    print(res.stdout, res.stderr)
    assert res.returncode == 0
    assert "abi_example: OK" in res.stdout
