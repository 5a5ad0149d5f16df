"""CPU oracle for the T-CSR build and the temporal neighbour sampler.

TEST INFRASTRUCTURE ONLY: tests, the smoke check and the benchmark's CPU
baseline leg may use this package; the product library never does.  It shares
no code with the GPU library.

``tgl_oracle.c`` holds the arithmetic (plain single-threaded C, built with
``-O2 -ffp-contract=off``); this module only marshals numpy arrays through
ctypes.  ``brute`` restates the same definitions as a linear scan over the raw
edge list, ``pointer`` replays the paper's chronological pointer advance; both
exist to pin the oracle.
"""
from __future__ import annotations

import ctypes as C
import math
import os
import subprocess
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tgl_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, EINVAL, ERANGE, ENOMEM = 0, -1, -2, -5
MODES = {"recent": 0, "most_recent": 0, "uniform": 1}

GCC_FLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
             "-fno-fast-math", "-Wall", "-Wextra"]


def compile_oracle(src: str = _SRC, out: str = _LIB, extra: Sequence[str] = ()) -> str:
    """Compile the oracle with gcc into a shared library and return its path."""
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.run(["gcc", *GCC_FLAGS, *extra, src, "-o", tmp, "-lm"], check=True)
    os.replace(tmp, out)
    return out


_lib_cache = {}


def load(path: Optional[str] = None) -> C.CDLL:
    """Load (building first if absent) the oracle library at ``path``."""
    path = path or _LIB
    if path in _lib_cache:
        return _lib_cache[path]
    if not os.path.exists(path):
        if path != _LIB:
            raise FileNotFoundError(path)
        compile_oracle()
    lib = C.CDLL(path)
    P = C.c_void_p
    i64, i32, u64, f32 = C.c_int64, C.c_int32, C.c_uint64, C.c_float
    lib.oracle_build.restype = i64
    lib.oracle_build.argtypes = [i64, P, P, P, P, i64, C.c_int, P, P, P, P]
    lib.oracle_locate_many.restype = None
    lib.oracle_locate_many.argtypes = [i64, P, P, i64, P, P, P, f32, P, P]
    lib.oracle_mix64.restype = u64
    lib.oracle_mix64.argtypes = [u64]
    lib.oracle_slot_hash.restype = u64
    lib.oracle_slot_hash.argtypes = [u64, u64, i32, i32, i32]
    lib.oracle_sample.restype = C.c_int
    lib.oracle_sample.argtypes = [i64, P, P, P, P, i64, P, P, i32, P, i32, i32, f32,
                                  u64, u64, P, P, P, P, P, P]
    lib.oracle_sample_anchored.restype = C.c_int
    lib.oracle_sample_anchored.argtypes = [i64, P, P, P, P, i64, P, P, i32, P, i32, i32, f32,
                                           u64, u64, i32, P, P, P, P, P, P]
    _lib_cache[path] = lib
    return lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


@dataclass
class TCSR:
    """Host T-CSR: indptr[N+1], and per entry nbr/eid/ts (structure of arrays)."""
    indptr: np.ndarray
    nbr: np.ndarray
    eid: np.ndarray
    ts: np.ndarray

    @property
    def num_nodes(self) -> int:
        return len(self.indptr) - 1


@dataclass
class Hop:
    nbr: np.ndarray
    eid: np.ndarray
    ts: np.ndarray
    dt: np.ndarray
    parent: Optional[np.ndarray]   # None for hop 1
    num_roots: int


class OracleError(RuntimeError):
    def __init__(self, status: int):
        super().__init__("oracle status %d" % status)
        self.status = status


def build_tcsr(src, dst, ts, eid, num_nodes: int, undirected: bool = True,
               lib: Optional[C.CDLL] = None) -> TCSR:
    lib = lib or load()
    src = np.ascontiguousarray(src, dtype=np.int32)
    dst = np.ascontiguousarray(dst, dtype=np.int32)
    ts = np.ascontiguousarray(ts, dtype=np.float32)
    eid = None if eid is None else np.ascontiguousarray(eid, dtype=np.int64)
    m0 = len(src)
    m = 2 * m0 if undirected else m0
    indptr = np.empty(num_nodes + 1, dtype=np.int64)
    nbr = np.empty(max(m, 1), dtype=np.int32)
    eo = np.empty(max(m, 1), dtype=np.int64)
    to = np.empty(max(m, 1), dtype=np.float32)
    r = lib.oracle_build(m0, _ptr(src), _ptr(dst), _ptr(ts), _ptr(eid), num_nodes,
                         int(bool(undirected)), _ptr(indptr), _ptr(nbr), _ptr(eo), _ptr(to))
    if r < 0:
        raise OracleError(int(r))
    return TCSR(indptr, nbr[:m], eo[:m], to[:m])


def locate(g: TCSR, x, t, s, delta: float, lib: Optional[C.CDLL] = None):
    """Candidate windows [lo, hi) of roots (x[i], t[i]) in snapshots s[i]."""
    lib = lib or load()
    x = np.ascontiguousarray(x, dtype=np.int32)
    t = np.ascontiguousarray(t, dtype=np.float32)
    s = np.ascontiguousarray(np.broadcast_to(np.asarray(s, dtype=np.int32), x.shape))
    lo = np.empty(len(x), dtype=np.int64)
    hi = np.empty(len(x), dtype=np.int64)
    lib.oracle_locate_many(g.num_nodes, _ptr(g.indptr), _ptr(g.ts), len(x), _ptr(x), _ptr(t),
                           _ptr(s), C.c_float(delta), _ptr(lo), _ptr(hi))
    return lo, hi


def mix64(z: int, lib: Optional[C.CDLL] = None) -> int:
    return int((lib or load()).oracle_mix64(C.c_uint64(z & (2**64 - 1))))


def slot_hash(seed: int, path: int, hop: int, s: int, j: int, lib: Optional[C.CDLL] = None) -> int:
    return int((lib or load()).oracle_slot_hash(seed & (2**64 - 1), path & (2**64 - 1), hop, s, j))


def capacities(num_roots: int, fanouts: Sequence[int], snapshots: int) -> List[int]:
    """Worst-case slots per hop: R*S*k1, then times k_h."""
    caps, c = [], num_roots * snapshots
    for k in fanouts:
        c *= k
        caps.append(c)
    return caps


ANCHORS = {"own": 0, "root": 1, 0: 0, 1: 1}


def sample(g: TCSR, roots, root_ts, fanouts: Sequence[int], mode: str = "uniform",
           snapshots: int = 1, snapshot_len: float = math.inf, seed: int = 0,
           root_base: int = 0, lib: Optional[C.CDLL] = None, anchor="own") -> List[Hop]:
    """Run Algorithm 1 serially; returns one ``Hop`` per layer, sliced to its size.
    ``anchor`` places the snapshot windows of hops >= 2: "own" (the root's own
    time) or "root" (the hop-1 root's time, below the root's own time)."""
    lib = lib or load()
    roots = np.ascontiguousarray(roots, dtype=np.int32)
    root_ts = np.ascontiguousarray(root_ts, dtype=np.float32)
    fan = np.ascontiguousarray(fanouts, dtype=np.int32)
    hops = len(fan)
    R = len(roots)
    caps = capacities(R, fanouts, snapshots)
    outs = [dict(nbr=np.empty(max(c, 1), np.int32), eid=np.empty(max(c, 1), np.int64),
                 ts=np.empty(max(c, 1), np.float32), dt=np.empty(max(c, 1), np.float32))
            for c in caps]
    parents = [None] + [np.empty(max(c, 1), np.int64) for c in caps[:-1]]
    PA = C.c_void_p * hops
    counts = np.zeros(hops, dtype=np.int64)
    r = lib.oracle_sample_anchored(g.num_nodes, _ptr(g.indptr), _ptr(g.nbr), _ptr(g.eid), _ptr(g.ts),
                          R, _ptr(roots), _ptr(root_ts), hops, _ptr(fan), MODES[mode],
                          snapshots, C.c_float(snapshot_len), seed & (2**64 - 1),
                          root_base & (2**64 - 1), ANCHORS[anchor],
                          PA(*[_ptr(o["nbr"]) for o in outs]), PA(*[_ptr(o["eid"]) for o in outs]),
                          PA(*[_ptr(o["ts"]) for o in outs]), PA(*[_ptr(o["dt"]) for o in outs]),
                          PA(*[_ptr(p) for p in parents]), _ptr(counts))
    if r != OK:
        raise OracleError(int(r))
    hops_out = []
    for h in range(hops):
        nr = int(counts[h])
        n = nr * (snapshots if h == 0 else 1) * int(fan[h])
        o = outs[h]
        hops_out.append(Hop(o["nbr"][:n], o["eid"][:n], o["ts"][:n], o["dt"][:n],
                            None if h == 0 else parents[h][:nr], nr))
    return hops_out
