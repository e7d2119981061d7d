"""Build libtreeverify.so (HIP kernels + C entry points) for gfx950, in-tree."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libtreeverify.so")
SOURCES = ["tv_api.hip", "tv_attention.hip", "tv_accept.hip", "tv_draft.hip", "tv_cache.hip",
           "tv_sample.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA results in VGPRs: the softmax reads the score tiles on the VALU,
    # so accumulation-register placement would add copies every tile
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    # inputs are finite by contract: fmax needs no NaN quieting
    "-fno-honor-nans",
    "-Wno-unused-command-line-argument",
    "-I" + os.path.join(ROOT, "include"),
]


def hipcc() -> str:
    for cand in [os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"]:
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False) -> str:
    """Compile every source into LIB (always rebuilds).  Returns the path."""
    tmp = LIB + ".tmp"
    cmd = [hipcc()] + HIPCC_FLAGS + [os.path.join(CSRC, s) for s in SOURCES] + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines()
                     if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + msgs)
    if verbose and msgs.strip():
        print(msgs)
    os.replace(tmp, LIB)
    return LIB


EXAMPLE_SRC = os.path.join(ROOT, "tests", "native", "abi_example.c")
EXAMPLE = os.path.join(ROOT, "tests", "native", "abi_example")


def build_example(verbose: bool = False, out: str = EXAMPLE) -> str:
    """Compile the plain-C program that drives the C ABI (a host-only build
    against libtreeverify.so and the HIP runtime)."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cmd = ["gcc", "-O2", "-std=c99", "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROOT, "include"),
           "-I" + os.path.join(rocm, "include"), EXAMPLE_SRC, "-o", out, "-L" + HERE,
           "-ltreeverify", "-L" + os.path.join(rocm, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath," + HERE + ":" + os.path.join(rocm, "lib")]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("gcc failed:\n" + res.stdout + res.stderr)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
