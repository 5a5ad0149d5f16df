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


def _ordered_bits(ts):
    """float32 -> int64 keys in [0, 2^32) with the order of the floats (no NaN)."""
    b = np.asarray(ts, np.float32).view(np.int32).astype(np.int64)
    return np.where(b >= 0, b | 0x80000000, (~b) & 0xFFFFFFFF)


def hist_of(indptr, nbr, ts):
    """The neighbour history of every entry, from its definition: positions
    [lo, hi) of the neighbour's run whose timestamps are below the entry's
    (lo = the run's start); (0, 0) for a neighbour outside the node range.
    Runs are sorted by time, so lo + #{run timestamps below t} is the lower
    bound of (neighbour, t) in the (owner, ts) order of all entries."""
    indptr = np.asarray(indptr, np.int64)
    nbr = np.asarray(nbr, np.int64)
    ts = np.asarray(ts, np.float32)
    n = len(indptr) - 1
    ok = (nbr >= 0) & (nbr < n)
    lo = np.zeros(len(nbr), np.int64)
    hi = np.zeros(len(nbr), np.int64)
    lo[ok] = indptr[nbr[ok]]
    owner = np.repeat(np.arange(n, dtype=np.int64), np.diff(indptr))
    key = (owner << 32) | _ordered_bits(ts)
    q = (nbr[ok] << 32) | _ordered_bits(ts[ok])
    order = np.argsort(q, kind="stable")      # sorted queries keep the search in cache
    pos = np.empty(len(q), np.int64)
    pos[order] = np.searchsorted(key, q[order], side="left")
    hi[ok] = pos
    return lo, hi


def check_hist_device(g, chunk=1 << 27):
    """Neighbour histories of a device T-CSR against their definition,
    computed on the device in chunks (for T-CSRs too large for the host)."""
    import torch
    M, n = g.num_entries, g.num_nodes
    ip = g.indptr

    def ordered(bits):
        bits = bits.long()
        return torch.where(bits >= 0, bits | 0x80000000, (~bits) & 0xFFFFFFFF)

    key = torch.repeat_interleave(torch.arange(n, device=ip.device, dtype=torch.int64), ip[1:] - ip[:-1],
                                  output_size=M) << 32
    for c0 in range(0, M, chunk):
        key[c0:c0 + chunk] |= ordered(g.ts[c0:c0 + chunk].view(torch.int32))
    words = g.entries.view(torch.int32)
    hs = g.hist
    for c0 in range(0, M, chunk):
        v = (words[c0:c0 + chunk, 0] & 0x7FFFFFFF).long()
        t = ordered(g.ts[c0:c0 + chunk].view(torch.int32))
        hi = torch.searchsorted(key, (v << 32) | t)
        got = hs[c0:c0 + chunk].long() & 0xFFFFFFFF
        assert torch.equal(got[:, 0], ip[v]), "neighbour history start differs in entries %d.." % c0
        assert torch.equal(got[:, 1], hi), "neighbour history end differs in entries %d.." % c0
    del key
    torch.cuda.empty_cache()


def dir_scale_np(f, l, K):
    """Cells per unit of time of runs with first and last timestamps f, l and
    K cells (tgl_cell): K / (l - f) in float32 when l - f is positive and
    finite, else 0."""
    f = np.asarray(f, np.float32)
    l = np.asarray(l, np.float32)
    with np.errstate(invalid="ignore", over="ignore", divide="ignore"):
        span = l - f
        ok = (span > 0) & np.isfinite(span)
        return np.where(ok, np.asarray(K).astype(np.float32) / np.where(ok, span, np.float32(1)),
                        np.float32(0)).astype(np.float32)


def dir_cell_np(t, f, l, sc, K):
    """The cell of time t in a run (tgl_cell): 0 for t <= f, K - 1 for t >= l,
    else min(K - 1, floor((t - f) * sc)), in float32 operations."""
    t = np.asarray(t, np.float32)
    f = np.asarray(f, np.float32)
    l = np.asarray(l, np.float32)
    sc = np.asarray(sc, np.float32)
    K = np.asarray(K, np.int64)
    with np.errstate(invalid="ignore", over="ignore"):
        x = (t - f) * sc
        mid = np.where(x < K.astype(np.float32), np.trunc(np.where(np.isfinite(x), x, 0)), K).astype(np.int64)
    mid = np.minimum(mid, K - 1)
    return np.where(~(t > f), 0, np.where(t >= l, K - 1, mid)).astype(np.int64)


def dir_cells(indptr, ts):
    """The time directory of every run, from its definition (tgl_cell): for
    search-index slot j, with a, b the run holding entry 32 j and k = j -
    ceil(a / 32) its cell, pos = a + #{entries of the run in cells below k} and
    its timestamp (+inf at b).  Cells grow along a run and runs follow each
    other, so slot ceil(a / 32) + cell is a non-decreasing key over all
    entries, and pos is the lower bound of j among the keys."""
    X = 32
    indptr = np.asarray(indptr, np.int64)
    ts = np.asarray(ts, np.float32)
    M = len(ts)
    L = -(-M // X)
    n = len(indptr) - 1
    a, b = indptr[:-1], indptr[1:]
    ja, jb = -(-a // X), -(-b // X)
    K = jb - ja
    has = b > a
    f = np.where(has, ts[np.minimum(a, max(M - 1, 0))] if M else np.inf, np.inf).astype(np.float32)
    l = np.where(has, ts[np.maximum(b - 1, 0)] if M else -np.inf, -np.inf).astype(np.float32)
    sc = dir_scale_np(f, l, K)
    owner = np.repeat(np.arange(n, dtype=np.int64), np.diff(indptr))
    c = dir_cell_np(ts, f[owner], l[owner], sc[owner], K[owner])
    key = np.where(K[owner] > 0, ja[owner] + c, ja[owner] - 1)
    assert np.all(np.diff(key) >= 0)
    j = np.arange(L, dtype=np.int64)
    pos = np.searchsorted(key, j, side="left")
    slot_owner = np.searchsorted(indptr, j * X, side="right") - 1
    end = indptr[slot_owner + 1]
    cts = np.full(L, np.inf, np.float32)
    inside = pos < end
    cts[inside] = ts[pos[inside]]
    return pos, cts


def check_dir_slots(g, chunk=1 << 24):
    """Time directory of a device T-CSR against its definition, slot by slot:
    with a, b, f, l the run of the entry 32 j (from the node records) and k
    its cell, pos must be the position where the run's cells reach k (entry
    pos - 1 in a lower cell or pos = a; entry pos in cell k or above, or pos
    = b), and the cell's timestamp that of entry pos (+inf at b).  Positions are gathered on the device;
    the cells are computed on the host in float32."""
    import torch
    M, n = g.num_entries, g.num_nodes
    L = -(-M // 32)
    ip = g.indptr
    rec = g.nodes[:, :4]
    for j0 in range(0, L, chunk):
        j = torch.arange(j0, min(L, j0 + chunk), device=ip.device, dtype=torch.int64)
        x = torch.searchsorted(ip, j * 32, right=True) - 1
        r = rec[x].cpu().numpy()
        d = g.dir[j0:j0 + len(j)]
        pos = d[:, 0].long() & 0xFFFFFFFF
        prev = ts_at(g.ts, pos - 1)
        here = ts_at(g.ts, pos)
        jn = j.cpu().numpy()
        pos = pos.cpu().numpy()
        a = r[:, 0].view(np.uint32).astype(np.int64)
        b = r[:, 1].view(np.uint32).astype(np.int64)
        f = r[:, 2].view(np.float32)
        l = r[:, 3].view(np.float32)
        assert np.all((a <= jn * 32) & (jn * 32 < b)), "node records do not cover the slots from %d" % j0
        ja = -(-a // 32)
        K = -(-b // 32) - ja
        k = jn - ja
        sc = dir_scale_np(f, l, K)
        assert np.all((pos >= a) & (pos <= b)), "directory position outside its run from slot %d" % j0
        cp = dir_cell_np(prev.cpu().numpy(), f, l, sc, K)
        ch = dir_cell_np(here.cpu().numpy(), f, l, sc, K)
        inside = pos < b
        assert np.all((pos == a) | (cp < k)), "directory position too high from slot %d" % j0
        assert np.all(~inside | (ch >= k)), "directory position too low from slot %d" % j0
        want = np.where(inside, here.cpu().numpy(), np.float32(np.inf)).astype(np.float32)
        got = d[:, 1].cpu().numpy().view(np.uint32)
        assert np.array_equal(got, want.view(np.uint32)), "directory timestamp from slot %d" % j0


def ts_at(ts, pos):
    """ts[pos] on the device, with positions clamped into the array."""
    import torch
    return ts[torch.clamp(pos, 0, ts.shape[0] - 1)]


def tcsr_to_host(g, hints=True, hist_on_host=True, dir_on_host=True):
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
    if g.dir is not None and dir_on_host and len(ts):
        pos, cts = dir_cells(ip, ts)
        d = g.dir.cpu().numpy().view(np.uint32)
        assert np.array_equal(d[:, 0].astype(np.int64), pos), "time directory positions: %d differ" % int(
            (d[:, 0] != pos).sum())
        assert np.array_equal(d[:, 1], cts.view(np.uint32)), "time directory timestamps"
    if g.hist is not None and hist_on_host:
        hs = g.hist.cpu().numpy().view(np.uint32).astype(np.int64)
        lo, hi = hist_of(ip, nbr, ts)
        assert np.array_equal(hs[:, 0], lo), "neighbour history start: %d differ" % int((hs[:, 0] != lo).sum())
        assert np.array_equal(hs[:, 1], hi), "neighbour history end: %d differ" % int((hs[:, 1] != hi).sum())
    return oracle.TCSR(g.indptr.cpu().numpy(), nbr.copy(), ent[:, 1].copy(),
                       w[:, 1].copy().view(np.float32))


def upload_oracle_tcsr(g):
    import paper_2203_14883_amd as P
    return P.tcsr_from_host(g.indptr, g.nbr, g.ts, g.eid)
