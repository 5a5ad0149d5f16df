"""Brute-force restatement of the sampler's definition, for tiny graphs.

TEST INFRASTRUCTURE ONLY.  It never builds a T-CSR: for every root and
snapshot it scans the raw edge list, keeps the entries owned by the root's node
whose timestamp lies in the window, orders them by (timestamp, input
position), and then applies the selection rule.  Pure Python loops, so use it
on graphs of at most a few thousand edges.  It shares nothing with
``tgl_oracle.c`` except the stated definition, which is why agreement between
the two pins the oracle's build, window search and selection.
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence

import numpy as np

M64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15


def mix64(z: int) -> int:
    """SplitMix64 finalizer (Steele, Lea & Flood, OOPSLA 2014), on Python ints."""
    z &= M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def slot_hash(seed: int, path: int, hop: int, s: int, j: int) -> int:
    key = (hop << 40) | (s << 24) | j
    return mix64(mix64(mix64((seed & M64) ^ GOLDEN) ^ (path & M64)) ^ key)


def _entries(src, dst, ts, eid, undirected):
    """Directed entries (owner, neighbour, time, edge id, input position)."""
    m0 = len(src)
    out = []
    for i in range(m0):
        e = i if eid is None else int(eid[i])
        t = float(np.float32(ts[i]))
        if t == 0.0:
            t = 0.0                       # -0 is stored as +0
        out.append((int(src[i]), int(dst[i]), t, e, i))
    if undirected:
        for i in range(m0):
            e = i if eid is None else int(eid[i])
            t = float(np.float32(ts[i]))
            if t == 0.0:
                t = 0.0
            out.append((int(dst[i]), int(src[i]), t, e, m0 + i))
    return out


def _window(t: float, s: int, delta: float):
    hi = t if s == 0 else t - s * delta
    lo = -math.inf if math.isinf(delta) else t - (s + 1) * delta
    return lo, hi


def _f32(x: float) -> np.float32:
    return np.float32(x)


def sample(src, dst, ts, eid, num_nodes: int, undirected: bool, roots, root_ts,
           fanouts: Sequence[int], mode: str, snapshots: int = 1,
           snapshot_len: float = math.inf, seed: int = 0, root_base: int = 0, anchor: str = "own"):
    """Returns a list of dicts per hop: nbr, eid, ts, dt (numpy) and parent.
    With anchor "root", a root of hop >= 2 takes the window s of its hop-1
    ancestor's time t0, cut below its own time t: t0 - (s+1)D <= ts < min(t0 - sD, t)."""
    ents = _entries(src, dst, ts, eid, undirected)
    by_owner = {}
    for en in ents:
        by_owner.setdefault(en[0], []).append(en)
    S = snapshots
    delta = float(np.float32(snapshot_len))
    # current roots: (node, time as float of f32, window, path, hop-1 ancestor time)
    cur = [(int(x), float(np.float32(t)), 0, (root_base + r) & M64, float(np.float32(t)))
           for r, (x, t) in enumerate(zip(roots, root_ts))]
    result = []
    for h, k in enumerate(fanouts, start=1):
        wins = S if h == 1 else 1
        nbr, eo, tso, dto, nxt, parent = [], [], [], [], [], []
        for q, (x, t, s_in, path, t0) in enumerate(cur):
            for w in range(wins):
                s = w if h == 1 else s_in
                if h >= 2 and anchor == "root":
                    lo, hi = _window(t0, s, delta)
                    hi = min(hi, t)
                else:
                    lo, hi = _window(t, s, delta)
                cands = []
                if 0 <= x < num_nodes:
                    cands = [en for en in by_owner.get(x, [])
                             if (en[2] >= lo) and (en[2] < hi)]
                cands.sort(key=lambda en: (en[2], en[4]))
                n = len(cands)
                for j in range(k):
                    slot = (q * wins + w) * k + j
                    pick = None
                    if mode in ("recent", "most_recent"):
                        if j < n:
                            pick = cands[n - 1 - j]
                    else:
                        if n > 0:
                            pick = cands[(slot_hash(seed, path, h, s, j) * n) >> 64]
                    if pick is None:
                        nbr.append(-1); eo.append(-1); tso.append(-1.0); dto.append(-1.0)
                        continue
                    _, v, te, e, _ = pick
                    nbr.append(v); eo.append(e); tso.append(te)
                    dto.append(float(_f32(t) - _f32(te)))    # float32 subtraction
                    if h < len(fanouts):
                        cpath = ((path * S * k + s * k + j) if h == 1 else (path * k + j)) & M64
                        nxt.append((v, te, s, cpath, t0))
                        parent.append(slot)
        result.append(dict(nbr=np.array(nbr, np.int32), eid=np.array(eo, np.int64),
                           ts=np.array(tso, np.float32), dt=np.array(dto, np.float32),
                           parent=None if h == 1 else np.array(prev_parent, np.int64),
                           num_roots=len(cur)))
        prev_parent = parent
        cur = nxt
    return result


def window_sizes(src, dst, ts, undirected: bool, num_nodes: int, x, t, s, delta):
    """Number of candidates of each (x, t, s) by a linear scan."""
    ents = _entries(src, dst, ts, None, undirected)
    d = float(np.float32(delta))
    out = []
    for xi, ti, si in zip(x, t, s):
        ti = float(np.float32(ti))
        lo, hi = _window(ti, int(si), d)
        if not 0 <= int(xi) < num_nodes:
            out.append(0)
            continue
        out.append(sum(1 for en in ents if en[0] == int(xi) and lo <= en[2] < hi))
    return np.array(out, np.int64)
