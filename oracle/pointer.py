"""Replay of the paper's pointer-based window location for layer 1.

TEST INFRASTRUCTURE ONLY.  Section 3.1 ("Sampling") and Algorithm 1 keep,
per node, one pointer per snapshot boundary into the node's time-sorted run
and advance them as the (chronological) roots arrive, so candidates are found
in O(1) amortised instead of by binary search.  This module implements that
mechanism independently of the oracle's binary search: for roots visited in
non-decreasing time order, boundary pointer i of node x sits at the first
entry with ts >= t - i*D (boundary 0 at t), and window s is
[pointer s+1, pointer s).  Agreement with ``oracle_locate`` pins the oracle's
search on layer 1.  Only finite root times and in-range nodes are meaningful
here (the paper's mechanism has no rule for others).
"""
from __future__ import annotations

import math

import numpy as np


def hop1_windows(indptr: np.ndarray, ts: np.ndarray, roots, root_ts,
                 snapshots: int, delta: float):
    """Returns (lo, hi) arrays of shape [R, S] from monotone pointer advances."""
    roots = np.asarray(roots)
    root_ts = np.asarray(root_ts, dtype=np.float32)
    R, S = len(roots), snapshots
    d = float(np.float32(delta))
    lo = np.zeros((R, S), np.int64)
    hi = np.zeros((R, S), np.int64)
    pointers = [dict() for _ in range(S + 1)]
    order = np.argsort(root_ts, kind="stable")
    for r in order:
        x = int(roots[r])
        t = float(root_ts[r])
        a, b = int(indptr[x]), int(indptr[x + 1])
        for i in range(S + 1):
            if i == 0:
                bound = t
            elif math.isinf(d):
                bound = -math.inf
            else:
                bound = t - i * d
            p = pointers[i].get(x, a)
            while p < b and float(ts[p]) < bound:
                p += 1
            pointers[i][x] = p
        for s in range(S):
            lo[r, s] = pointers[s + 1][x]
            hi[r, s] = pointers[s][x]
    return lo, hi
