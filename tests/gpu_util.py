"""Helpers for GPU tests: device checks, uploads and host copies."""
import sys

import numpy as np
import pytest

import oracle


def announce(msg):
    """Names the case about to run on the GPU (flushed, so a fault still shows it)."""
    print("[gpu-case] " + msg, flush=True)
    sys.stdout.flush()


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch


def upload(a, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a if dtype is None else np.asarray(a, dtype)))
    return t.cuda()


def hops_to_numpy(hops):
    return [dict(nbr=h.nbr.cpu().numpy(), eid=h.eid.cpu().numpy(), ts=h.ts.cpu().numpy(),
                 dt=h.dt.cpu().numpy(), parent=None if h.parent is None else h.parent.cpu().numpy(),
                 num_roots=h.num_roots) for h in hops]


def first_hints(indptr, nbr, ts):
    """The neighbour-first hint of every entry, from its definition: the
    neighbour's run (sorted by time) has no timestamp below the entry's, i.e.
    the neighbour's first timestamp (+inf for an empty run) is not below it.
    Neighbour ids outside the node range get no hint."""
    indptr = np.asarray(indptr, np.int64)
    nbr = np.asarray(nbr, np.int64)
    ts = np.asarray(ts, np.float32)
    n = len(indptr) - 1
    first = np.full(n, np.inf, np.float32)
    ne = indptr[1:] > indptr[:-1]
    first[ne] = ts[indptr[:-1][ne]]
    ok = (nbr >= 0) & (nbr < n)
    h = np.zeros(len(nbr), bool)
    h[ok] = ~(first[nbr[ok]] < ts[ok])
    return h


def tcsr_to_host(g, hints=True):
    """Host copy of a device T-CSR; checks that the separate timestamp array
    equals the records' timestamps bit for bit, and that the neighbour-first
    hint bits follow their definition (or, with hints=False, are all clear)."""
    ent = g.entries.cpu().numpy().reshape(-1, 2)
    w = ent.view(np.int32).reshape(-1, 4)
    ts = g.ts.cpu().numpy()
    assert np.array_equal(ts.view(np.int32), w[:, 1]), "ts array differs from the records"
    ip = g.indptr.cpu().numpy()
    nbr = w[:, 0] & 0x7FFFFFFF
    got_hint = w[:, 0] < 0
    want_hint = first_hints(ip, nbr, ts) if hints else np.zeros(len(nbr), bool)
    assert np.array_equal(got_hint, want_hint), "neighbour-first hints: %d of %d differ" % (
        int((got_hint != want_hint).sum()), len(nbr))
    nodes = g.nodes.cpu().numpy()
    assert np.array_equal(nodes[:, 0].view(np.uint32), ip[:-1]), "node summary start"
    assert np.array_equal(nodes[:, 1].view(np.uint32), ip[1:]), "node summary end"
    nonempty = ip[1:] > ip[:-1]
    first = np.where(nonempty, ts[np.minimum(ip[:-1], max(len(ts) - 1, 0))] if len(ts) else np.inf, np.inf).astype(np.float32)
    last = np.where(nonempty, ts[np.maximum(ip[1:] - 1, 0)] if len(ts) else -np.inf, -np.inf).astype(np.float32)
    assert np.array_equal(nodes[:, 2].view(np.float32).view(np.uint32), first.view(np.uint32)), "node summary first ts"
    assert np.array_equal(nodes[:, 3].view(np.float32).view(np.uint32), last.view(np.uint32)), "node summary last ts"
    assert nodes.shape[1] == 32
    for i in range(28):                     # inline timestamps of each run's first 28 entries
        has = ip[:-1] + i < ip[1:]
        want = np.full(len(has), np.inf, np.float32)
        want[has] = ts[ip[:-1][has] + i]
        assert np.array_equal(nodes[:, 4 + i].view(np.uint32), want.view(np.uint32)), "inline ts %d" % i
    if g.ts_index is not None:
        tsx = g.ts_index.cpu().numpy()
        assert np.array_equal(tsx.view(np.uint32), ts[::32].view(np.uint32)), "search index"
    return oracle.TCSR(g.indptr.cpu().numpy(), nbr.copy(), ent[:, 1].copy(),
                       w[:, 1].copy().view(np.float32))


def upload_oracle_tcsr(g):
    import paper_2203_14883_amd as P
    return P.tcsr_from_host(g.indptr, g.nbr, g.ts, g.eid)
