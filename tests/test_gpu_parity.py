"""GPU path (through the C ABI) against the CPU oracle, bit for bit.

Every comparison is on the same seeded inputs: the T-CSR built on the GPU
must equal the oracle's T-CSR, and sampling on the GPU must equal the
oracle's sampling (nbr, eid, float32 ts and dt bit patterns, parent indices,
per-hop root counts)."""
import dataclasses
import math

import numpy as np
import pytest

import oracle
import paper_2203_14883_amd as P
from paper_2203_14883_amd import workloads as W
from checks import assert_hops_equal, same_bits, first_diff
from gpu_util import announce, hops_to_numpy, require_gpu, tcsr_to_host, upload, upload_oracle_tcsr

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    return require_gpu()


def assert_tcsr_equal(got, want, what=""):
    assert np.array_equal(got.indptr, want.indptr), what + " indptr: " + str(first_diff(got.indptr, want.indptr))
    assert same_bits(got.nbr, want.nbr), what + " nbr: " + str(first_diff(got.nbr, want.nbr))
    assert same_bits(got.eid, want.eid), what + " eid: " + str(first_diff(got.eid, want.eid))
    assert same_bits(got.ts, want.ts), what + " ts: " + str(first_diff(got.ts, want.ts))


def gpu_build(src, dst, ts, eid, n, undirected, hist=True, dir=True):
    return P.tcsr_build(upload(src, np.int32), upload(dst, np.int32), upload(ts, np.float32),
                        None if eid is None else upload(eid, np.int64), n, undirected, hist=hist, dir=dir)


def gpu_sample(g, roots, rts, fan, mode, S, D, seed, base, anchor="own"):
    out = P.sample(g, upload(roots, np.int32), upload(rts, np.float32), fan, mode, S, D, seed, base,
                   anchor=anchor)
    return hops_to_numpy(out)


def _rand_case(rng):
    N = int(rng.integers(1, 60))
    m0 = int(rng.integers(0, 600))
    src = rng.integers(0, N, m0).astype(np.int32)
    dst = rng.integers(0, N, m0).astype(np.int32)
    ts = rng.integers(-5, 40, m0).astype(np.float32)
    if m0:
        ts[rng.integers(0, m0, max(1, m0 // 8))] = -0.0
        ts[rng.integers(0, m0, max(1, m0 // 50))] = np.float32(rng.choice([np.inf, -np.inf, 1e-42, -3.5]))
    und = bool(rng.integers(0, 2))
    eid = None if rng.integers(0, 2) else rng.integers(-10, 2**40, m0).astype(np.int64)
    R = int(rng.integers(0, 300))
    roots = rng.integers(-2, N + 2, R).astype(np.int32)
    rts = rng.integers(-5, 45, R).astype(np.float32)
    if R > 6:
        rts[:6] = [np.nan, np.inf, -np.inf, -0.0, 1e-41, 3.25]
    hops = int(rng.integers(1, 5))
    choices = [1, 2, 5, 10, 16, 33, 70] if hops <= 2 else [1, 2, 3, 5]
    fan = [int(rng.choice(choices)) for _ in range(hops)]
    mode = ["recent", "uniform"][int(rng.integers(0, 2))]
    S = int(rng.choice([1, 1, 2, 3, 5]))
    D = float(rng.choice([1.0, 2.5, 9.0])) if (S > 1 or rng.integers(0, 2)) else math.inf
    return N, src, dst, ts, eid, und, roots, rts, fan, mode, S, D, int(rng.integers(0, 2**63)), int(rng.integers(0, 2**62))


def test_random_small_graphs(torch):
    """GPU build and GPU sampling on random small graphs with ties, -0, +-inf and
    denormal timestamps, self-loops, duplicate / out-of-range roots, NaN and
    infinite query times, 1-4 hops, fanouts 1..70 and 1..5 snapshots."""
    rng = np.random.default_rng(2024)
    for trial in range(160):
        N, src, dst, ts, eid, und, roots, rts, fan, mode, S, D, seed, base = _rand_case(rng)
        hist = trial % 3 != 2              # with and without neighbour histories
        tdir = trial % 4 != 3              # with and without time directories
        announce("random trial %d N=%d m0=%d R=%d fan=%s mode=%s S=%d D=%s hist=%s dir=%s"
                 % (trial, N, len(src), len(roots), fan, mode, S, D, hist, tdir))
        want_g = oracle.build_tcsr(src, dst, ts, eid, N, und)
        g = gpu_build(src, dst, ts, eid, N, und, hist, tdir)
        assert_tcsr_equal(tcsr_to_host(g), want_g, "trial %d" % trial)
        want = oracle.sample(want_g, roots, rts, fan, mode, S, D, seed, base)
        got = gpu_sample(g, roots, rts, fan, mode, S, D, seed, base)
        assert_hops_equal(got, want, "trial %d" % trial)
        for h in range(len(fan)):
            assert got[h]["num_roots"] == want[h].num_roots


PRESETS = [
    ("c1", {}, None),
    ("c2", {}, "all"),
    ("c3", dict(num_nodes=16_682, num_edges=2_000_000, t_buckets=17_000), [0, 1, 117, 250, 499]),
    ("c4", dict(num_nodes=1_000_000, num_edges=10_700_000), [0, 1, 1000, 2000, 2674]),
    ("c5", dict(num_nodes=1_000_000, num_edges=10_000_000, batch_edges=60_000), [0, 1, 80, 166]),
]


@pytest.fixture(scope="module")
def preset_cache():
    return {}


def _preset(name, kw, cache):
    if name not in cache:
        w = W.make(name, **kw)
        src, dst, ts, eid = w.build_input()
        cache[name] = (w, oracle.build_tcsr(src, dst, ts, eid, w.num_nodes, w.undirected))
    return cache[name]


@pytest.mark.parametrize("name,kw,batches", PRESETS, ids=[p[0] for p in PRESETS])
def test_preset_build_parity(torch, name, kw, batches, preset_cache):
    w, want = _preset(name, kw, preset_cache)
    src, dst, ts, eid = w.build_input()
    announce("build %s nodes=%d edges=%d" % (name, w.num_nodes, w.num_edges))
    g = gpu_build(src, dst, ts, eid, w.num_nodes, w.undirected)
    torch.cuda.synchronize()
    assert_tcsr_equal(tcsr_to_host(g), want, name)


@pytest.mark.parametrize("name,kw,batches", PRESETS, ids=[p[0] for p in PRESETS])
def test_preset_sample_parity(torch, name, kw, batches, preset_cache):
    """Sampling on the oracle's T-CSR uploaded as-is, so a sampler bug cannot
    hide behind a build bug."""
    w, g_host = _preset(name, kw, preset_cache)
    g = upload_oracle_tcsr(g_host)
    if batches is None:
        groups = [list(w.default_batches)]
    elif batches == "all":
        groups = [list(range(w.num_batches()))]
    else:
        groups = [[b] for b in batches] + [list(batches[:2])]
    for grp in groups:
        roots = np.concatenate([w.batch(b)[0] for b in grp])
        rts = np.concatenate([w.batch(b)[1] for b in grp])
        base = w.root_base(grp[0]) if grp == list(range(grp[0], grp[0] + len(grp))) else None
        if base is None:      # non-consecutive batches: sample each with its own base
            continue
        announce("sample %s batches %s..%s roots=%d" % (name, grp[0], grp[-1], len(roots)))
        want = oracle.sample(g_host, roots, rts, w.fanouts, w.mode, w.snapshots, w.snapshot_len,
                             w.sample_seed, base)
        got = gpu_sample(g, roots, rts, w.fanouts, w.mode, w.snapshots, w.snapshot_len,
                         w.sample_seed, base)
        assert_hops_equal(got, want, "%s batches %s" % (name, grp))


def test_batching_invariance_and_determinism(torch):
    w = W.make_c2()
    g = gpu_build(w.src, w.dst, w.ts, None, w.num_nodes, True)
    roots, rts, base = w.batches(10, 30)
    announce("c2 batches 10..29 in one call")
    whole = gpu_sample(g, roots, rts, w.fanouts, "uniform", 1, math.inf, 7, base)
    again = gpu_sample(g, roots, rts, w.fanouts, "uniform", 1, math.inf, 7, base)
    assert_hops_equal(again, whole, "repeat")
    parts = []
    for b in range(10, 30):
        r, t, bb = w.batch(b)
        parts.append(gpu_sample(g, r, t, w.fanouts, "uniform", 1, math.inf, 7, bb))
    for h in range(2):
        for f in ("nbr", "eid", "ts", "dt"):
            cat = np.concatenate([p[h][f] for p in parts])
            assert same_bits(whole[h][f], cat), (h, f)


def test_build_range_errors(torch):
    ok = np.array([0, 1, 2], np.int32)
    t = np.array([1, 2, 3], np.float32)
    for src, dst, ts in [(np.array([0, 3, 1], np.int32), ok, t), (ok, np.array([0, -1, 1], np.int32), t),
                         (ok, ok, np.array([1, np.nan, 2], np.float32))]:
        for und in (False, True):
            announce("build range error und=%s" % und)
            with pytest.raises(P.TglError) as e:
                gpu_build(src, dst, ts, None, 3, und)
            assert e.value.status == -2


def test_build_key_layouts(torch):
    """Sort keys of both forms: packed (node field, timestamp field and
    neighbour id in 64 bits, the neighbour below the sort digits) and plain
    (node << 32 | timestamp key), fields with no varying bit (one owner, one
    timestamp, one node), timestamp fields of 1, 8 and 10 bits (the
    neighbours' first timestamps then compared as 8- or 16-bit fields), ties on
    every key, and graphs with more nodes than twice the entries, whose hints
    are set after the node records."""
    rng = np.random.default_rng(1234)
    N20 = 1 << 20
    cases = []
    for und in (False, True):
        m0 = 3000
        cases += [
            ("plain: random float ts, N=2^20", N20, rng.integers(0, N20, m0), rng.integers(0, N20, m0),
             rng.uniform(-1e6, 1e6, m0), und),
            ("packed: years, N=2^20", N20, rng.integers(0, N20, m0), rng.integers(0, N20, m0),
             rng.integers(1900, 2022, m0), und),
            ("packed: one owner", 5000, np.full(m0, 77), rng.integers(0, 5000, m0), rng.integers(0, 50, m0), und),
            ("packed: one timestamp", 5000, rng.integers(0, 5000, m0), rng.integers(0, 5000, m0),
             np.full(m0, 3.5), und),
            ("packed: one node", 1, np.zeros(m0), np.zeros(m0), rng.integers(0, 9, m0), und),
            ("packed: 10-bit timestamp field", 5000, rng.integers(0, 5000, m0), rng.integers(0, 5000, m0),
             rng.integers(1024, 2048, m0), und),
            ("packed: 1-bit timestamp field", 700, rng.integers(0, 700, m0), rng.integers(0, 700, m0),
             rng.choice([6.0, 7.0], m0), und),
            ("plain: one owner, random ts", N20, np.full(m0, N20 - 1), rng.integers(0, N20, m0),
             rng.uniform(-1e30, 1e30, m0), und),
            ("packed: N > 2M", 4000, rng.integers(0, 4000, 300), rng.integers(0, 4000, 300),
             rng.integers(0, 20, 300), und),
            ("plain: N > 2M", N20, rng.integers(0, N20, 300), rng.integers(0, N20, 300),
             rng.uniform(0, 1e8, 300), und),
        ]
    for what, N, src, dst, ts, und in cases:
        src, dst, ts = src.astype(np.int32), dst.astype(np.int32), ts.astype(np.float32)
        eid = rng.integers(0, 2**40, len(src)).astype(np.int64) if und else None
        announce("key layout: %s und=%s" % (what, und))
        want = oracle.build_tcsr(src, dst, ts, eid, N, und)
        g = gpu_build(src, dst, ts, eid, N, und)
        assert_tcsr_equal(tcsr_to_host(g), want, "%s und=%s" % (what, und))


def test_degenerate_cases(torch):
    # empty graph: every root PAD; zero roots; single-node graph with a self-loop
    announce("empty graph")
    g = gpu_build(np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), None, 4, True)
    assert g.indptr.cpu().tolist() == [0, 0, 0, 0, 0]
    out = gpu_sample(g, np.array([0, 3, 9], np.int32), np.array([1, 2, 3], np.float32), [4, 2],
                     "uniform", 1, math.inf, 1, 0)
    assert np.all(out[0]["nbr"] == -1) and out[1]["num_roots"] == 0
    announce("zero roots")
    g = gpu_build(np.array([0], np.int32), np.array([0], np.int32), np.array([5], np.float32), None, 1, True)
    out = gpu_sample(g, np.zeros(0, np.int32), np.zeros(0, np.float32), [3, 3], "recent", 2, 4.0, 1, 0)
    assert out[0]["num_roots"] == 0 and out[1]["num_roots"] == 0
    announce("self loop")
    out = gpu_sample(g, np.array([0, 0], np.int32), np.array([6, 5], np.float32), [3], "recent", 1, math.inf, 1, 0)
    assert out[0]["nbr"].tolist() == [0, 0, -1, -1, -1, -1]


def test_long_runs_and_off_grid_window_edges(torch):
    """Runs whose lengths straddle the inline timestamps of a node record (27-29)
    and the held-stretch sizes of the 8-, 16-, 32- and 64-lane searches (61/62,
    125/126, 253/254) plus long runs, timestamps on a
    1/16 grid near 1e6 with ties, and window lengths (0.1, 0.37) whose edges
    t - i*delta fall between adjacent float32 values; 1..64 snapshots, so the
    edges of a root are located in batches with ragged last batches."""
    rng = np.random.default_rng(77)
    lens = [200_000, 61, 62, 125, 126, 253, 254, 5_000, 1, 27, 28, 29, 4]
    N = len(lens) + 1                     # the last node has no entries
    src = np.concatenate([np.full(L, x, np.int32) for x, L in enumerate(lens)])
    dst = rng.integers(0, N, len(src)).astype(np.int32)
    ts = np.concatenate([np.float32(1e6) + np.float32(0.0625) * rng.integers(0, max(2, L // 3), L).astype(np.float32)
                         for L in lens]).astype(np.float32)
    want_g = oracle.build_tcsr(src, dst, ts, None, N, False)
    g = gpu_build(src, dst, ts, None, N, False)
    assert_tcsr_equal(tcsr_to_host(g), want_g, "long runs")
    assert g.ts_index is not None and g.dir is not None
    variants = ((g, "directory and index"), (dataclasses.replace(g, dir=None), "index"),
                (dataclasses.replace(g, ts_index=None), "directory"),
                (dataclasses.replace(g, ts_index=None, dir=None), "neither"))
    for S, D, R in [(1, math.inf, 3000), (1, 0.1, 3000), (3, 0.37, 3000), (7, 0.1, 1500), (8, 0.37, 1500),
                    (9, 0.1, 1000), (64, 0.1, 300)]:
        roots = rng.integers(0, N, R).astype(np.int32)
        span = np.float32(0.0625) * np.float32(70_000)
        rts = (np.float32(1e6) + rng.random(R, dtype=np.float32) * span).astype(np.float32)
        rts[: R // 3] = ts[rng.integers(0, len(ts), R // 3)]          # query times equal to timestamps
        # one hop most recent: the last window's lower edge comes from the
        # gathered entries' timestamps instead of a search
        for mode, fan in (("recent", [10, 5]), ("uniform", [10, 5]), ("recent", [10])):
            announce("long runs S=%d D=%s R=%d mode=%s fan=%s" % (S, D, R, mode, fan))
            want = oracle.sample(want_g, roots, rts, fan, mode, S, D, 11, 3)
            for gg, what in variants:
                got = gpu_sample(gg, roots, rts, fan, mode, S, D, 11, 3)
                assert_hops_equal(got, want, "S=%d D=%s %s %s %s" % (S, D, mode, fan, what))


def test_guided_search_on_skewed_runs(torch):
    """The first round on the search index places its probes by interpolating
    between a run's first and last timestamps, and the time directory splits
    the same span into even cells; the window edges must not depend on how
    well either fits the run.  Long runs (indexed search) whose
    timestamps are far from evenly spread -- nearly all at the start, nearly
    all at the end, geometric, two clusters, one value with two outliers, one
    value throughout, and an even spread for contrast -- queried at entry timestamps, between them
    and outside the run, with 1-3 snapshots and 1-2 hops."""
    rng = np.random.default_rng(4242)
    L = 60_000
    runs = [
        np.sort(rng.random(L) * 1e6),                                           # even
        np.sort(np.where(rng.random(L) < 0.98, rng.random(L), 1e6 * rng.random(L))),   # piled at the start
        np.sort(np.where(rng.random(L) < 0.98, 1e6 - rng.random(L), 1e6 * rng.random(L))),   # piled at the end
        np.sort(2.0 ** (rng.random(L) * 40.0)),                                 # geometric over 12 decades
        np.sort(np.concatenate([rng.random(L // 2) * 10.0, 9.9e5 + rng.random(L - L // 2) * 10.0])),  # two clusters
        np.concatenate([[-1e9], np.full(L - 2, 5.0), [1e9]]),                   # one value, two outliers
        np.full(L, 5.0),                                                        # one value throughout
    ]
    N = len(runs)
    src = np.concatenate([np.full(L, x, np.int32) for x in range(N)])
    dst = rng.integers(0, N, len(src)).astype(np.int32)
    ts = np.concatenate(runs).astype(np.float32)
    want_g = oracle.build_tcsr(src, dst, ts, None, N, False)
    g = gpu_build(src, dst, ts, None, N, False)
    assert_tcsr_equal(tcsr_to_host(g), want_g, "skewed runs")
    R = 4000
    roots = rng.integers(0, N, R).astype(np.int32)
    rts = ts[rng.integers(0, len(ts), R)].copy()                                 # equal to timestamps
    rts[R // 4: R // 2] = np.nextafter(rts[R // 4: R // 2], np.float32(np.inf))  # just above them
    rts[R // 2: 3 * R // 4] = (rng.random(R // 4) * 2e6 - 5e5).astype(np.float32)   # anywhere, also outside
    rts[3 * R // 4:] = np.float32(2.0) ** rng.integers(0, 41, R - 3 * R // 4).astype(np.float32)
    for S, D in [(1, math.inf), (1, 3e4), (3, 1e3), (3, 2.5)]:
        for mode, fan in (("recent", [10]), ("uniform", [10, 3])):
            announce("skewed runs S=%d D=%s mode=%s" % (S, D, mode))
            want = oracle.sample(want_g, roots, rts, fan, mode, S, D, 5, 0)
            for gg, what in ((g, "directory"), (dataclasses.replace(g, dir=None), "index")):
                got = gpu_sample(gg, roots, rts, fan, mode, S, D, 5, 0)
                assert_hops_equal(got, want, "skewed runs S=%d D=%s %s %s" % (S, D, mode, what))


def test_column_view_round_trip(torch):
    """The column layout of Sec. 3.1 (indptr, nbr, ts, eid as separate arrays)
    in and out of the entries on the device: columns unpacked from a GPU
    build equal the oracle's; the oracle's columns packed on the device give
    the same T-CSR (records, index, hints, histories, directories against
    their definitions) and the same samples, with and without edge ids."""
    rng = np.random.default_rng(31)
    for trial in range(12):
        N, src, dst, ts, eid, und, roots, rts, fan, mode, S, D, seed, base = _rand_case(rng)
        if trial == 0:
            src, dst, ts, eid = src[:0], dst[:0], ts[:0], None
        announce("columns trial %d N=%d m0=%d eid=%s" % (trial, N, len(src), eid is not None))
        og = oracle.build_tcsr(src, dst, ts, eid, N, und)
        g = gpu_build(src, dst, ts, eid, N, und)
        nbr, e = P.tcsr_columns(g)
        assert np.array_equal(nbr.cpu().numpy(), og.nbr.astype(np.int32)), "unpacked nbr, trial %d" % trial
        assert np.array_equal(e.cpu().numpy(), og.eid), "unpacked eid, trial %d" % trial
        pos_ids = trial % 2 == 1                     # pack without edge ids: eid = position
        h = P.tcsr_from_columns(upload(og.indptr, np.int64), upload(og.nbr, np.int32), upload(og.ts, np.float32),
                                None if pos_ids else upload(og.eid, np.int64))
        want_g = og if not pos_ids else oracle.TCSR(og.indptr, og.nbr, np.arange(len(og.nbr), dtype=np.int64), og.ts)
        assert_tcsr_equal(tcsr_to_host(h), want_g, "columns trial %d" % trial)
        want = oracle.sample(want_g, roots, rts, fan, mode, S, D, seed, base)
        assert_hops_equal(gpu_sample(h, roots, rts, fan, mode, S, D, seed, base), want, "columns trial %d" % trial)


def test_chunk_scheduled_batches(torch):
    """Batches of random chunk scheduling (Alg. 2) -- edge ranges that start at
    chunk offsets, not at the batch grid -- fused into one GPU call, against the
    oracle on the same roots and root_base."""
    w = W.make_c2(n_users=3000, n_items=400, num_edges=60_000, seed=8)
    og = oracle.build_tcsr(w.src, w.dst, w.ts, None, w.num_nodes, True)
    g = gpu_build(w.src, w.dst, w.ts, None, w.num_nodes, True)
    for epoch in (0, 3):
        sch = w.chunk_schedule(epoch, 150)
        parts = [w.edge_batch(a, b, epoch) for a, b in sch[10:16]]
        roots = np.concatenate([p[0] for p in parts])
        rts = np.concatenate([p[1] for p in parts])
        base = parts[0][2]
        announce("chunk-scheduled batches epoch %d start %d" % (epoch, sch[0][0]))
        want = oracle.sample(og, roots, rts, (10, 10), "uniform", 1, math.inf, epoch, base)
        got = gpu_sample(g, roots, rts, (10, 10), "uniform", 1, math.inf, epoch, base)
        assert_hops_equal(got, want, "epoch %d" % epoch)


def test_snapshot_anchor_root(torch):
    """Snapshot anchor A (windows of hops >= 2 at the hop-1 root's time, cut
    below the root's own time) on random graphs with 2-4 hops, several
    snapshots and finite window lengths, and on a reduced c5 (3 snapshots of
    1e6, 2-hop uniform)."""
    rng = np.random.default_rng(99)
    trial = 0
    while trial < 60:
        N, src, dst, ts, eid, und, roots, rts, fan, mode, S, D, seed, base = _rand_case(rng)
        if len(fan) < 2:
            continue
        if math.isinf(D):
            S, D = int(rng.integers(2, 5)), float(rng.choice([2.5, 9.0]))
        trial += 1
        announce("anchor trial %d N=%d m0=%d R=%d fan=%s mode=%s S=%d D=%s" % (trial, N, len(src), len(roots), fan,
                                                                              mode, S, D))
        want_g = oracle.build_tcsr(src, dst, ts, eid, N, und)
        g = gpu_build(src, dst, ts, eid, N, und)
        want = oracle.sample(want_g, roots, rts, fan, mode, S, D, seed, base, anchor="root")
        got = gpu_sample(g, roots, rts, fan, mode, S, D, seed, base, anchor="root")
        assert_hops_equal(got, want, "anchor trial %d" % trial)
    w = W.make_c5(num_nodes=1_000_000, num_edges=10_000_000, batch_edges=60_000)
    og = oracle.build_tcsr(w.src, w.dst, w.ts, None, w.num_nodes, True)
    g = P.tcsr_from_host(og.indptr, og.nbr, og.ts, og.eid)
    roots, rts, base = w.batches(80, 81)
    for anchor in ("root", "own"):
        announce("anchor %s on reduced c5" % anchor)
        want = oracle.sample(og, roots, rts, w.fanouts, w.mode, w.snapshots, w.snapshot_len, w.sample_seed, base,
                             anchor=anchor)
        got = gpu_sample(g, roots, rts, w.fanouts, w.mode, w.snapshots, w.snapshot_len, w.sample_seed, base,
                         anchor=anchor)
        assert_hops_equal(got, want, "c5 anchor %s" % anchor)


def test_neighbour_first_hints(torch):
    """The neighbour-first hint (bit 31 of a T-CSR entry's nbr) lets a later
    hop skip the node record of a root with an empty window, and the
    neighbour history (per entry, its neighbour's entries older than it)
    gives a later hop's window outright when windows are unbounded below.
    Samples must be the oracle's with the hints set exactly or clear
    everywhere, with and without histories, and with either snapshot anchor,
    on random graphs of 2-4 hops (directed and undirected, with finite and
    infinite windows) and on a reduced c4, where about half of the hop-2
    roots carry the hint."""
    rng = np.random.default_rng(31)
    trial = 0
    while trial < 40:
        N, src, dst, ts, eid, und, roots, rts, fan, mode, S, D, seed, base = _rand_case(rng)
        if len(fan) < 2:
            continue
        trial += 1
        anchor = "root" if trial % 3 == 0 and not math.isinf(D) else "own"
        announce("hint trial %d N=%d m0=%d R=%d fan=%s mode=%s S=%d D=%s anchor=%s"
                 % (trial, N, len(src), len(roots), fan, mode, S, D, anchor))
        og = oracle.build_tcsr(src, dst, ts, eid, N, und)
        want = oracle.sample(og, roots, rts, fan, mode, S, D, seed, base, anchor=anchor)
        for hints, hist in ((True, True), (True, False), (False, False), (False, True)):
            g = P.tcsr_from_host(og.indptr, og.nbr, og.ts, og.eid, hints=hints, hist=hist)
            what = "hint trial %d (hints=%s, hist=%s)" % (trial, hints, hist)
            assert_tcsr_equal(tcsr_to_host(g, hints=hints), og, what)
            got = gpu_sample(g, roots, rts, fan, mode, S, D, seed, base, anchor=anchor)
            assert_hops_equal(got, want, what)
    w = W.make_c4(num_nodes=1_000_000, num_edges=10_700_000)
    og = oracle.build_tcsr(w.src, w.dst, w.ts, None, w.num_nodes, True)
    roots, rts, base = w.batches(2000, 2008)
    want = oracle.sample(og, roots, rts, w.fanouts, w.mode, w.snapshots, w.snapshot_len, w.sample_seed, base)
    # hop-2 roots whose entry carries the hint: the path is exercised
    first = np.full(w.num_nodes, np.inf, np.float32)
    ne = og.indptr[1:] > og.indptr[:-1]
    first[ne] = og.ts[og.indptr[:-1][ne]]
    v = want[0].nbr >= 0
    hinted = ~(first[want[0].nbr[v]] < want[0].ts[v])
    assert hinted.mean() > 0.3, "reduced c4: only %.2f of the hop-2 roots are hinted" % hinted.mean()
    for hints, hist in ((True, True), (True, False), (False, False), (False, True)):
        announce("hints=%s hist=%s on reduced c4" % (hints, hist))
        g = P.tcsr_from_host(og.indptr, og.nbr, og.ts, og.eid, hints=hints, hist=hist)
        got = gpu_sample(g, roots, rts, w.fanouts, w.mode, w.snapshots, w.snapshot_len, w.sample_seed, base)
        assert_hops_equal(got, want, "reduced c4 (hints=%s, hist=%s)" % (hints, hist))


def test_many_windows(torch):
    """First hops with 2-12 snapshot windows on either side of the switch
    between the multi-window kernel (up to 8 windows, window edges held in
    LDS) and the wide one (more windows), both modes, 1-3 hops, with long
    runs (searched on the index) and short ones (node-record timestamps)."""
    rng = np.random.default_rng(77)
    N = 40
    lens = [30_000, 2_000, 300, 61, 28, 5] + [int(x) for x in rng.integers(0, 50, N - 6)]
    src = np.concatenate([np.full(L, x, np.int32) for x, L in enumerate(lens)])
    dst = rng.integers(0, N, len(src)).astype(np.int32)
    ts = rng.integers(0, 20_000, len(src)).astype(np.float32)
    og = oracle.build_tcsr(src, dst, ts, None, N, True)
    g = P.tcsr_from_host(og.indptr, og.nbr, og.ts, og.eid)
    for trial, S in enumerate((2, 7, 8, 9, 12)):
        for mode in ("recent", "uniform"):
            fan = [(3, 2), (5,), (2, 2, 2)][(trial + (mode == "uniform")) % 3]
            D = float(rng.choice([250.0, 1000.0, 1500.5]))
            R = 700
            roots = rng.integers(-1, N + 1, R).astype(np.int32)
            rts = rng.integers(0, 21_000, R).astype(np.float32)
            seed, base = int(rng.integers(0, 2**62)), int(rng.integers(0, 2**40))
            announce("many windows S=%d mode=%s fan=%s D=%s" % (S, mode, fan, D))
            want = oracle.sample(og, roots, rts, fan, mode, S, D, seed, base)
            got = gpu_sample(g, roots, rts, fan, mode, S, D, seed, base)
            assert_hops_equal(got, want, "S=%d %s" % (S, mode))
