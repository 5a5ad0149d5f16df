"""Pins of the feature / state lookup oracle (oracle/features.py) against
things other than itself:

* the same definition as an explicit per-slot loop;
* a closed form: a table whose row r holds the value r everywhere turns the
  lookup into "key where valid, 0 elsewhere";
* the edge-feature rows of sampled slots equal the slots' own eids, and the
  node rows their nbr (a table encoding its row index), on the sampler oracle's
  output for a seeded graph;
* plausible mistakes (clamping keys, no zero rows, off-by-one bound, wrong key
  array, ignoring the limit) each fail one of these checks.
"""
import numpy as np
import pytest

import oracle
from oracle import features as F
from paper_2203_14883_amd import workloads as W


def _random_case(rng, n=200):
    nbr = rng.integers(-1, 60, n).astype(np.int32)
    eid = rng.integers(-1, 90, n).astype(np.int64)
    nbr[:3] = [-1, 49, 50]          # PAD, last row, first key past a 50-row table
    eid[:3] = [80, -1, 79]
    tables = [(rng.standard_normal((50, 12)).astype(np.float32), F.NODE),
              (rng.integers(-100, 100, (80, 3, 8)).astype(np.int16), F.EDGE),
              (rng.standard_normal((0, 4)).astype(np.float32), F.NODE),
              (rng.integers(0, 255, (50, 16)).astype(np.uint8), F.NODE)]
    return nbr, eid, tables


def _pin_checks(gather):
    rng = np.random.default_rng(3)
    # 1. explicit loop
    nbr, eid, tables = _random_case(rng)
    for lim in (None, 0, 17, 10**6):
        got = gather(nbr, eid, tables, lim)
        want = F.gather_loop(nbr, eid, tables, lim)
        for g, w in zip(got, want):
            if g.shape != w.shape or g.dtype != w.dtype or g.tobytes() != w.tobytes():
                return False
    # 2. closed form on an index-encoding table
    rows = np.repeat(np.arange(40, dtype=np.int64)[:, None], 5, axis=1)
    keys = rng.integers(-3, 45, 300).astype(np.int64)
    (out,) = gather(None, keys, [(rows, F.EDGE)])
    want = np.where((keys >= 0) & (keys < 40), keys, 0)[:, None].repeat(5, axis=1)
    if not np.array_equal(out, want):
        return False
    (out,) = gather(keys.astype(np.int32), None, [(rows, F.NODE)], 100)
    if out.shape != (100, 5) or not np.array_equal(out, want[:100]):
        return False
    return True


def test_gather_pins():
    assert _pin_checks(F.gather)


def _clamp(nbr, eid, tables, limit=None):
    outs = []
    for rows, key in tables:
        k = np.asarray(nbr if key == F.NODE else eid, np.int64)
        n = len(k) if limit is None else max(0, min(int(limit), len(k)))
        k = np.clip(k[:n], 0, max(rows.shape[0] - 1, 0))
        outs.append(rows[k] if rows.shape[0] else np.zeros((n,) + rows.shape[1:], rows.dtype))
    return outs


def _no_zero(nbr, eid, tables, limit=None):
    outs = F.gather(nbr, eid, tables, limit)
    return [np.full_like(o, 7) if o.size else o for o in outs]   # invalid rows left as garbage


def _off_by_one(nbr, eid, tables, limit=None):
    outs = []
    for rows, key in tables:
        k = np.asarray(nbr if key == F.NODE else eid, np.int64)
        n = len(k) if limit is None else max(0, min(int(limit), len(k)))
        k = k[:n]
        out = np.zeros((n,) + rows.shape[1:], rows.dtype)
        ok = (k >= 0) & (k <= rows.shape[0] - 2)
        out[ok] = rows[k[ok]]
        outs.append(out)
    return outs


def _wrong_key(nbr, eid, tables, limit=None):
    swapped = [(r, F.EDGE if k == F.NODE else F.NODE) for r, k in tables]
    if nbr is None or eid is None:
        return F.gather(nbr, eid, tables, limit)
    return F.gather(nbr, eid.astype(np.int32), swapped, limit)


def _no_limit(nbr, eid, tables, limit=None):
    return F.gather(nbr, eid, tables, None)


@pytest.mark.parametrize("mutant", [_clamp, _no_zero, _off_by_one, _wrong_key, _no_limit])
def test_gather_pins_catch_mutants(mutant):
    assert not _pin_checks(mutant)


def test_gathered_rows_of_sampled_slots():
    """Rows looked up for the sampler oracle's slots: an edge table encoding
    edge ids returns each slot's eid, a node table encoding node ids its nbr;
    PAD slots give zeros."""
    w = W.make_c2(n_users=300, n_items=40, num_edges=4000, seed=9)
    g = oracle.build_tcsr(w.src, w.dst, w.ts, None, w.num_nodes, True)
    roots, rts, base = w.batches(1, 4)
    hops = oracle.sample(g, roots, rts, (10, 10), "uniform", 1, float("inf"), 3, base)
    erows = np.repeat(np.arange(w.num_edges, dtype=np.int64)[:, None], 2, axis=1)
    nrows = np.repeat(np.arange(w.num_nodes, dtype=np.int32)[:, None], 4, axis=1)
    for h in hops:
        ef, nf = F.gather(h.nbr, h.eid, [(erows, F.EDGE), (nrows, F.NODE)])
        pad = h.nbr < 0
        assert np.array_equal(ef[:, 0], np.where(pad, 0, h.eid))
        assert np.array_equal(nf[:, 3], np.where(pad, 0, h.nbr))
        assert pad.any() and (~pad).any()
