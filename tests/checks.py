"""Shared comparison and invariant helpers for oracle and GPU tests."""
import math

import numpy as np

PAD_F32_BITS = np.float32(-1.0).view(np.uint32)


def same_bits(a, b):
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    return a.shape == b.shape and a.dtype == b.dtype and np.array_equal(a.view(np.uint8), b.view(np.uint8))


def first_diff(a, b):
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    if a.shape != b.shape:
        return "shape %s vs %s" % (a.shape, b.shape)
    ne = np.nonzero((a.view(np.uint8).reshape(len(a), -1) != b.view(np.uint8).reshape(len(b), -1)).any(axis=1))[0]
    if len(ne) == 0:
        return None
    i = int(ne[0])
    return "first of %d differences at %d: %r vs %r" % (len(ne), i, a[i], b[i])


def assert_hops_equal(got, want, what=""):
    """Bitwise equality of every field of every hop (objects with nbr/eid/ts/dt/parent)."""
    assert len(got) == len(want), what
    for h, (g, w) in enumerate(zip(got, want)):
        for f in ("nbr", "eid", "ts", "dt"):
            a, b = _field(g, f), _field(w, f)
            assert same_bits(a, b), "%s hop %d field %s: %s" % (what, h + 1, f, first_diff(a, b))
        if h > 0:
            a, b = _field(g, "parent"), _field(w, "parent")
            assert same_bits(a, b), "%s hop %d parent: %s" % (what, h + 1, first_diff(a, b))


def _field(o, f):
    return o[f] if isinstance(o, dict) else getattr(o, f)


def check_invariants(g, roots, root_ts, hops, fanouts, mode, S, delta):
    """Properties any correct output has, checked against the host T-CSR ``g``."""
    roots = np.asarray(roots)
    root_ts = np.asarray(root_ts, np.float32)
    d = float(np.float32(delta))
    # per-hop roots (node, time, window)
    cur_x, cur_t = roots.astype(np.int64), root_ts
    cur_s = np.zeros(len(roots), np.int64)
    for h, (hop, k) in enumerate(zip(hops, fanouts)):
        wins = S if h == 0 else 1
        n_roots = len(cur_x)
        nbr = hop.nbr.reshape(n_roots, wins, k)
        ts = hop.ts.reshape(n_roots, wins, k)
        dt = hop.dt.reshape(n_roots, wins, k)
        eid = hop.eid.reshape(n_roots, wins, k)
        valid = nbr >= 0
        # PAD slots carry -1 in every field
        assert np.all(eid[~valid] == -1)
        assert np.all(ts[~valid].view(np.uint32) == PAD_F32_BITS)
        assert np.all(dt[~valid].view(np.uint32) == PAD_F32_BITS)
        t = cur_t[:, None, None]
        s = cur_s[:, None, None] if h > 0 else np.arange(wins)[None, :, None]
        with np.errstate(invalid="ignore"):
            hi = np.where(s == 0, t.astype(np.float64), t.astype(np.float64) - s * d)
            lo = np.full(hi.shape, -np.inf) if math.isinf(d) else t.astype(np.float64) - (s + 1) * d
        tsd = ts.astype(np.float64)
        # strictly older than the root, inside the snapshot window
        assert np.all((tsd < hi)[valid]), "slot not older than the window top"
        assert np.all((tsd >= lo)[valid]), "slot below the window bottom"
        # dt is the float32 difference
        want_dt = (t.astype(np.float32) - ts).astype(np.float32)
        assert np.array_equal(dt[valid].view(np.uint32), np.broadcast_to(want_dt, dt.shape)[valid].view(np.uint32))
        assert np.all(dt[valid] > 0)
        # valid slots form a prefix of each group
        first_pad = np.where(valid, 0, 1).cumsum(axis=2)
        assert np.all(~valid | (first_pad == 0)), "valid slots are not a prefix"
        cnt = valid.sum(axis=2)
        if mode == "recent":
            # newest first: non-increasing timestamps
            dif = np.diff(np.where(valid, tsd, 0.0), axis=2)
            vv = valid[:, :, 1:]
            assert np.all(dif[vv] <= 0)
        else:
            assert np.all((cnt == 0) | (cnt == k)), "uniform group partly filled"
        # every valid slot is an entry of the root's node in the host T-CSR
        xs = np.broadcast_to(cur_x[:, None, None], nbr.shape)[valid]
        if len(xs):
            a = g.indptr[xs]
            b = g.indptr[xs + 1]
            # find each (nbr, eid, ts) inside the run: check membership via a sample
            idx = np.arange(len(xs))
            pick = idx if len(idx) <= 2000 else np.random.default_rng(0).choice(idx, 2000, replace=False)
            vn, ve, vt = nbr[valid], eid[valid], ts[valid]
            for i in pick:
                run = slice(int(a[i]), int(b[i]))
                m = (g.nbr[run] == vn[i]) & (g.eid[run] == ve[i]) & (g.ts[run].view(np.uint32) == vt[i].view(np.uint32))
                assert m.any(), "slot is not an entry of its root's run"
        if h + 1 < len(hops):
            nxt = hops[h + 1]
            flat_valid = valid.reshape(-1)
            want_parent = np.nonzero(flat_valid)[0]
            assert np.array_equal(nxt.parent, want_parent)
            assert np.all(np.diff(nxt.parent) > 0)
            cur_x = hop.nbr[want_parent].astype(np.int64)
            cur_t = hop.ts[want_parent]
            w_of = (want_parent // k) % wins if h == 0 else cur_s[want_parent // k]
            cur_s = w_of.astype(np.int64)
