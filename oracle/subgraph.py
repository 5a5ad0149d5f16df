"""Owned-entry extraction: the part of a temporal graph the oracle needs.

TEST INFRASTRUCTURE ONLY.  The oracle builds its T-CSR on the host with a
plain sort, which cannot hold billion-edge graphs.  Sampling a set of roots
only reads the runs of the nodes the sample reaches, so for checks at full
size the oracle builds a T-CSR of exactly those runs: the forward entries of
edges whose source is in the node set, then the reversed entries of edges
whose destination is in the set, each kept in input order.  Built without the
undirected flag, this gives every node of the set the same run, in the same
tie order, as the full undirected T-CSR (entry positions differ, which the
sampler never exposes).
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle


def owned_entries(src, dst, ts, eid, num_nodes, nodes, undirected=True, threads=16):
    """(src, dst, ts, eid) of the directed entries owned by ``nodes``."""
    flag = np.zeros(num_nodes, dtype=bool)
    flag[np.asarray(nodes, dtype=np.int64)] = True
    n = len(src)
    fwd = np.empty(n, dtype=bool)
    rev = np.empty(n, dtype=bool)
    chunk = 1 << 24

    def f(c):
        b, e = c * chunk, min(n, (c + 1) * chunk)
        np.take(flag, src[b:e], out=fwd[b:e])
        np.take(flag, dst[b:e], out=rev[b:e])

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(f, range((n + chunk - 1) // chunk)))
    fi = np.flatnonzero(fwd)
    ri = np.flatnonzero(rev) if undirected else np.zeros(0, np.int64)
    e_all = np.arange(n, dtype=np.int64) if eid is None else np.asarray(eid, np.int64)
    return (np.concatenate([src[fi], dst[ri]]).astype(np.int32),
            np.concatenate([dst[fi], src[ri]]).astype(np.int32),
            np.concatenate([ts[fi], ts[ri]]).astype(np.float32),
            np.concatenate([e_all[fi], e_all[ri]]))


def owned_tcsr(src, dst, ts, eid, num_nodes, nodes, undirected=True):
    """Oracle T-CSR holding the full runs of ``nodes`` (other runs partial)."""
    s, d, t, e = owned_entries(src, dst, ts, eid, num_nodes, nodes, undirected)
    return oracle.build_tcsr(s, d, t, e, num_nodes, False)


def reach_tcsr(src, dst, ts, eid, num_nodes, undirected, roots, root_ts, fanouts, mode,
               snapshots, snapshot_len, seed, root_base):
    """Oracle T-CSR with the full run of every node the sampling of ``roots``
    reaches (the roots, then the neighbours the oracle itself draws at each hop
    but the last)."""
    reach = np.unique(np.asarray(roots, np.int64))
    reach = reach[(reach >= 0) & (reach < num_nodes)]
    g = owned_tcsr(src, dst, ts, eid, num_nodes, reach, undirected)
    for h in range(len(fanouts) - 1):
        out = oracle.sample(g, roots, root_ts, fanouts[:h + 1], mode, snapshots, snapshot_len,
                            seed, root_base)
        nb = out[h].nbr[out[h].nbr >= 0]
        reach = np.unique(np.concatenate([reach, nb.astype(np.int64)]))
        g = owned_tcsr(src, dst, ts, eid, num_nodes, reach, undirected)
    return g
