"""Compiles libtgl.so (HIP, gfx950) in the package directory.

Usage: ``python -m paper_2203_14883_amd.build_lib`` or ``build()``.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

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
    # bit-exact float arithmetic: no FMA contraction, no flush of denormals
    "-ffp-contract=off",
    "-fno-gpu-flush-denormals-to-zero",
    # never emit packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed (%d): %s" % (r.returncode, cmd[-1]))
    if verbose and (r.stdout or r.stderr):
        sys.stderr.write(_filter(r.stdout + r.stderr))


def build(verbose: bool = False, out: str = LIB, extra=()) -> str:
    """Compiles every source to an object file (in parallel, one hipcc per
    source) and links them into ``out``."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tag = ".tmp%d" % os.getpid()
    objs = []
    cmds = []
    for src in sources():
        obj = os.path.join(os.path.dirname(out), os.path.basename(src) + tag + ".o")
        objs.append(obj)
        cmds.append([hipcc, *HIPCC_FLAGS, *extra, "-I", INCLUDE, "-I", CSRC, "-c", src, "-o", obj])
    tmp = out + tag
    try:
        jobs = max(1, min(len(cmds), int(os.environ.get("MAX_JOBS", "8"))))
        with ThreadPoolExecutor(jobs) as ex:
            list(ex.map(lambda c: _run(c, verbose), cmds))
        _run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
        os.replace(tmp, out)
    finally:
        for f in objs + [tmp]:
            if os.path.exists(f):
                os.remove(f)
    return out


def _filter(text: str) -> str:
    # the host pass does not know the packed-fp32 feature and says so once per file
    return "".join(l + "\n" for l in text.splitlines() if "packed-fp32-ops" not in l)


if __name__ == "__main__":
    print(build(verbose=True))
