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

and of the time encoding (Eq. 3) against closed forms (omega = 0, dt = 0,
omega * dt a multiple of pi) and a 50-digit mpmath evaluation at Wikipedia-
sized time differences, with its own mutants (sin for cos, phi dropped, a
float32 argument, PAD rows encoded).
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


# ---------------------------------------------------------------------------
# time encoding (Eq. 3)
# ---------------------------------------------------------------------------

def _te_pin_checks(enc):
    """Pins of the time encoding against closed forms and an independent
    50-digit evaluation (mpmath)."""
    import mpmath
    f32 = np.float32
    # closed forms: omega = 0 gives cos(phi); dt = 0 likewise; phi = 0 and
    # omega * dt = 0 gives 1; PAD rows are zero
    phi = np.array([0.0, np.pi / 3, np.pi / 2, np.pi, -np.pi / 3], f32)
    want_phi = np.array([1.0, 0.5, 0.0, -1.0, 0.5])
    out = enc(np.array([0.0, 5.0, -1.0], f32), np.array([0.0, 0.0, 0.0, 0.0, 0.0], f32), phi)
    if out.shape != (3, 5) or np.abs(out[0] - want_phi).max() > 1e-7 or np.abs(out[1] - want_phi).max() > 1e-7:
        return False
    if np.any(out[2] != 0.0):
        return False
    # omega = 1/1024 and dt a multiple of 1024 * pi in float: omega * dt = k * pi
    # up to dt's float rounding, so the value is +-1 to first order
    out = enc(np.array([f32(1024 * np.pi * 3)], f32), np.array([1.0 / 1024], f32), np.array([0.0], f32))
    if abs(out[0, 0] + 1.0) > 1e-6:
        return False
    # large arguments (Wikipedia-sized dt): against mpmath at 50 digits
    rng = np.random.default_rng(4)
    dt = (rng.random(64) * 2.7e6).astype(f32)
    omega = (1.0 / 10 ** np.linspace(0, 9, 16)).astype(f32)   # the TGAT-style frequency ladder
    phi = (rng.random(16) * 6.0 - 3.0).astype(f32)
    out = enc(dt, omega, phi)
    mpmath.mp.dps = 50
    for i in range(0, 64, 7):
        for j in range(16):
            exact = float(mpmath.cos(mpmath.mpf(float(omega[j])) * mpmath.mpf(float(dt[i])) + mpmath.mpf(float(phi[j]))))
            if abs(out[i, j] - exact) > 1e-9:
                return False
    # limit
    if enc(dt, omega, phi, 5).shape != (5, 16) or enc(dt, omega, phi, 0).shape != (0, 16):
        return False
    return True


def test_time_encode_pins():
    assert _te_pin_checks(F.time_encode)


def _te_sin(dt, omega, phi, limit=None):
    out = F.time_encode(dt, omega, phi, limit)
    d = np.asarray(dt, np.float32)[:out.shape[0]].astype(np.float64)[:, None]
    s = np.sin(d * np.asarray(omega, np.float64)[None, :] + np.asarray(phi, np.float64)[None, :])
    return np.where(out == 0.0, 0.0, s)


def _te_no_phi(dt, omega, phi, limit=None):
    return F.time_encode(dt, omega, np.zeros_like(np.asarray(phi)), limit)


def _te_float32_argument(dt, omega, phi, limit=None):
    dt = np.asarray(dt, np.float32)
    n = len(dt) if limit is None else max(0, min(int(limit), len(dt)))
    a = (dt[:n, None] * np.asarray(omega, np.float32)[None, :] + np.asarray(phi, np.float32)[None, :]).astype(np.float32)
    out = np.cos(a.astype(np.float64))
    out[~(dt[:n] >= 0)] = 0.0
    return out


def _te_pad_not_zero(dt, omega, phi, limit=None):
    dt = np.abs(np.asarray(dt, np.float32))
    return F.time_encode(dt, omega, phi, limit)


@pytest.mark.parametrize("mutant", [_te_sin, _te_no_phi, _te_float32_argument, _te_pad_not_zero])
def test_time_encode_pins_catch_mutants(mutant):
    assert not _te_pin_checks(mutant)
