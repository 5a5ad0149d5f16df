"""Compiles libtgl.so (HIP, gfx950) in the package directory.

Usage: ``python -m paper_2203_14883_amd.build_lib`` or ``build()``.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libtgl.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # bit-exact float arithmetic: no FMA contraction, no flush of denormals
    "-ffp-contract=off",
    "-fno-gpu-flush-denormals-to-zero",
    # never emit packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def build(verbose: bool = False, out: str = LIB, extra=()) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [hipcc, *HIPCC_FLAGS, *extra, "-I", INCLUDE, "-I", CSRC, *sources(), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed (%d)" % r.returncode)
    if verbose and (r.stdout or r.stderr):
        sys.stderr.write(_filter(r.stdout + r.stderr))
    os.replace(tmp, out)
    return out


def _filter(text: str) -> str:
    # the host pass does not know the packed-fp32 feature and says so once per file
    return "".join(l + "\n" for l in text.splitlines() if "packed-fp32-ops" not in l)


if __name__ == "__main__":
    print(build(verbose=True))
