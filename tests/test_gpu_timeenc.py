"""tgl_time_encode (through the C ABI) against the Eq. 3 oracle.

Tolerance, from the arithmetic: the kernel forms the argument in turns,
(omega / 2 pi) dt + phi / 2 pi, in double (within 5e-8 rad of exact below
2^24 turns; beyond, a double cosine), takes its fraction exactly, rounds the
folded fraction to float (2.4e-8 rad) and sums a cosine series to the x^12
term (6.4e-9 left out) in float (a few ulp of a value in [-1, 1]): within
3e-7 of cos(omega dt + phi).  So float32 rows are within 1e-6 of the float64
oracle; bfloat16 rows add the final rounding, at most half a bfloat16 ulp of
a value below 1 in magnitude (2^-9).  PAD rows must be exactly zero."""
import math

import numpy as np
import pytest

import oracle
from oracle import features as F
import paper_2203_14883_amd as P
from paper_2203_14883_amd import workloads as W
from gpu_util import announce, require_gpu

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-6
TOL_BF16 = 2.0 ** -9 + 1e-6


@pytest.fixture(scope="module")
def torch():
    return require_gpu()


def _host(torch, t):
    return t.float().cpu().numpy().astype(np.float64)


def _check(got, want, tol, what):
    pad = np.all(want == 0.0, axis=1) if want.size else np.zeros(0, bool)
    assert np.array_equal(np.isnan(got), np.isnan(want)), what + ": NaN pattern"
    ok = ~np.isnan(want)
    err = np.abs(got[ok] - want[ok])
    assert err.size == 0 or err.max() <= tol, "%s: max error %.3g > %.3g" % (what, err.max(), tol)
    assert np.all(got[pad] == 0.0), what + ": PAD rows not zero"


def test_random_encodings(torch):
    rng = np.random.default_rng(21)
    for trial in range(40):
        n = int(rng.choice([0, 1, 3, 4, 5, 63, 64, 65, 1000, 20000]))
        dim = int(rng.choice([1, 7, 64, 65, 100, 172, 4096] if n <= 1000 else [1, 100, 172]))
        dt = (rng.random(n) * float(rng.choice([10.0, 2.7e6, 1e8]))).astype(np.float32)
        if n >= 6:
            dt[:6] = [-1.0, 0.0, 1e-42, -1.0, np.float32(1e8), np.inf]
        if rng.integers(0, 2):
            omega = (1.0 / 10 ** np.linspace(0, 9, dim)).astype(np.float32)
        else:
            omega = (rng.standard_normal(dim) * float(rng.choice([1e-3, 1.0]))).astype(np.float32)
        phi = (rng.random(dim) * 6.0 - 3.0).astype(np.float32)
        use_count = bool(rng.integers(0, 2))
        per = int(rng.integers(1, 4))
        cval = int(rng.integers(-1, n // per + 3)) if use_count else None
        limit = None if cval is None else max(0, min(n, cval * per))
        m = n if limit is None else limit
        for odt, tol in ((torch.float32, TOL_F32), (torch.bfloat16, TOL_BF16)):
            announce("time encode trial %d n=%d dim=%d count=%s per=%d out=%s" % (trial, n, dim, cval, per, odt))
            out = torch.full((n, dim), 7.0, dtype=odt, device="cuda")
            count = None if cval is None else torch.tensor([cval], dtype=torch.int64, device="cuda")
            P.time_encode(torch.from_numpy(dt).cuda(), torch.from_numpy(omega).cuda(), torch.from_numpy(phi).cuda(),
                          out_dtype=odt, count=count, per_count=per, out=out)
            with np.errstate(invalid="ignore"):
                want = F.time_encode(dt, omega, phi, limit)
            got = _host(torch, out)
            _check(got[:m], want, tol, "trial %d %s" % (trial, odt))
            assert np.all(got[m:] == 7.0), "trial %d: rows past the count written" % trial


def test_encode_sampled_slots(torch):
    """Time encoding (100 dims, TGL's default) of every hop of a GPU sampling
    call on a Wikipedia-shaped graph, limited on the device to each hop's valid
    prefix, against the oracle's encoding of the oracle's own samples."""
    w = W.make_c2(n_users=2000, n_items=300, num_edges=40_000, seed=17)
    og = oracle.build_tcsr(w.src, w.dst, w.ts, None, w.num_nodes, True)
    g = P.tcsr_from_host(og.indptr, og.nbr, og.ts, og.eid)
    roots, rts, base = w.batches(2, 8)
    fan = (10, 10)
    dim = 100
    omega = (1.0 / 10 ** np.linspace(0, 9, dim)).astype(np.float32)
    phi = np.zeros(dim, np.float32)
    d_w, d_p = torch.from_numpy(omega).cuda(), torch.from_numpy(phi).cuda()
    for mode, S, D in (("uniform", 1, math.inf), ("recent", 2, 5.0e4)):
        announce("time encoding of sampled slots mode=%s S=%d" % (mode, S))
        smp = P.Sampler(len(roots), fan, S)
        smp.run(g, torch.from_numpy(roots).cuda(), torch.from_numpy(rts).cuda(), mode, D, 6, base)
        want_hops = oracle.sample(og, roots, rts, fan, mode, S, D, 6, base)
        for h, k in enumerate(fan):
            cap = smp.caps[h + 1]
            out = torch.full((cap, dim), 7.0, device="cuda")
            P.time_encode(smp.dt[h], d_w, d_p, n=cap, count=smp.counts[h:h + 1],
                          per_count=k * (S if h == 0 else 1), out=out)
            wh = want_hops[h]
            m = len(wh.dt)
            got = _host(torch, out)
            _check(got[:m], F.time_encode(wh.dt, omega, phi), TOL_F32, "hop %d" % (h + 1))
            assert np.all(got[m:] == 7.0), "hop %d: rows past the hop written" % (h + 1)
