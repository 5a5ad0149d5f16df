"""The seeded input generators: deterministic, chronological, and shaped like
the presets they stand in for (Table 3 of the paper gives the dataset shapes)."""
import math

import numpy as np
import pytest

from paper_2203_14883_amd import workloads as W

SMALL = {
    "c1": {},
    "c2": {},
    "c3": dict(num_nodes=1000, num_edges=300_000, t_buckets=3_000),
    "c4": dict(num_nodes=300_000, num_edges=3_000_000),
    "c5": dict(num_nodes=100_000, num_edges=1_000_000),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_deterministic_and_chronological(name):
    a = W.make(name, **SMALL[name])
    b = W.make(name, **SMALL[name])
    for f in ("src", "dst", "ts"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    assert a.src.dtype == np.int32 and a.dst.dtype == np.int32 and a.ts.dtype == np.float32
    assert np.all(np.diff(a.ts) >= 0)
    assert a.src.min() >= 0 and a.src.max() < a.num_nodes
    assert a.dst.min() >= 0 and a.dst.max() < a.num_nodes
    r1, t1, base1 = a.batch(a.num_batches() - 1)
    r2, t2, base2 = b.batch(b.num_batches() - 1)
    assert np.array_equal(r1, r2) and np.array_equal(t1, t2) and base1 == base2


def test_full_size_small_presets():
    c1 = W.make_c1()
    assert (c1.num_nodes, c1.num_edges) == (2000, 20_000)
    assert c1.src.max() < 1000 and c1.dst.min() >= 1000
    roots, ts, base = c1.batch(c1.default_batches[0])
    assert len(roots) == 200 and np.array_equal(roots[:100], c1.src[-100:])
    assert np.all(ts == np.concatenate([c1.ts[-100:]] * 2))
    assert np.all(c1.ts == np.floor(c1.ts))
    c2 = W.make_c2()
    assert (c2.num_nodes, c2.num_edges, c2.num_batches()) == (9227, 157_474, 263)
    assert len(c2.batch(262)[0]) == 3 * (157_474 - 262 * 600)
    neg = c2.negatives_of(5)
    assert neg.min() >= 8227 and neg.max() < 9227
    assert c2.ts.max() < 2.7e6


def test_c4_shape():
    w = W.make_c4(num_nodes=400_000, num_edges=4_272_000)
    years = w.ts
    assert years.min() >= 1900 and years.max() <= 2020 and np.all(years == np.floor(years))
    # citing paper's year is never earlier than the cited paper's year
    year_of = np.full(w.num_nodes, np.nan, np.float32)
    year_of[w.src] = w.ts
    cited = year_of[w.dst]
    known = ~np.isnan(cited)
    assert np.all(cited[known] <= w.ts[known])
    deg = np.bincount(w.src, minlength=w.num_nodes)
    assert deg.sum() == 4_272_000 and abs(deg.mean() - 10.68) < 1e-6


def test_c5_build_order_is_a_permutation():
    w = W.make_c5(num_nodes=10_000, num_edges=100_000)
    src, dst, ts, eid = w.build_input()
    assert np.array_equal(np.sort(eid), np.arange(w.num_edges))
    assert np.array_equal(src, w.src[eid]) and np.array_equal(ts, w.ts[eid])
    assert not np.all(np.diff(ts) >= 0)
    assert w.snapshots == 3 and w.snapshot_len == 1e6 and not math.isinf(w.snapshot_len)


def test_chunk_schedule_alg2():
    """Random chunk scheduling (Alg. 2): each epoch's batches start at a chunk
    boundary inside the first batch, are contiguous, all full, and stop before
    running past the last edge; the start moves from epoch to epoch."""
    w = W.make_c2(n_users=500, n_items=60, num_edges=10_000, seed=3)
    bs, cs = w.batch_edges, 50
    starts = set()
    for epoch in range(20):
        sch = w.chunk_schedule(epoch, cs)
        e_s = sch[0][0]
        assert 0 <= e_s < bs and e_s % cs == 0
        starts.add(e_s)
        for (a, b), (c, d) in zip(sch, sch[1:]):
            assert b == c
        assert all(b - a == bs for a, b in sch)
        assert sch[-1][1] <= w.num_edges < sch[-1][1] + bs
        assert w.chunk_schedule(epoch, cs) == sch          # deterministic per epoch
    assert len(starts) > 3
    # one chunk per batch: the schedule is the aligned batch grid (whole batches only)
    assert w.chunk_schedule(7, bs) == [(b * bs, (b + 1) * bs) for b in range(w.num_edges // bs)]
    with pytest.raises(ValueError):
        w.chunk_schedule(0, 7)


def test_edge_batch_matches_aligned_batches():
    w = W.make_c2(n_users=500, n_items=60, num_edges=10_000, seed=3)
    bs = w.batch_edges
    for b in (0, 3, 9):
        r, t, base = w.batch(b)
        r2, t2, base2 = w.edge_batch(b * bs, (b + 1) * bs, epoch=1)
        assert base2 == base
        assert np.array_equal(r2[:2 * bs], r[:2 * bs]) and np.array_equal(t2, t)
        assert r2[2 * bs:].min() >= w.neg_range[0] and r2[2 * bs:].max() < w.neg_range[1]


def test_chunk_batches_fuse_like_aligned_batches():
    """Consecutive chunk-scheduled batches sampled in one call (root_base of
    the first) give the same slots as sampled one by one: their root indices
    are disjoint and contiguous."""
    import oracle
    w = W.make_c2(n_users=500, n_items=60, num_edges=10_000, seed=3)
    g = oracle.build_tcsr(w.src, w.dst, w.ts, None, w.num_nodes, True)
    sch = w.chunk_schedule(4, 100)[5:8]
    parts = [w.edge_batch(a, b, epoch=4) for a, b in sch]
    roots = np.concatenate([p[0] for p in parts])
    rts = np.concatenate([p[1] for p in parts])
    whole = oracle.sample(g, roots, rts, (10, 10), "uniform", 1, math.inf, 11, parts[0][2])
    one = [oracle.sample(g, r, t, (10, 10), "uniform", 1, math.inf, 11, base) for r, t, base in parts]
    for h in range(2):
        assert np.array_equal(whole[h].nbr, np.concatenate([o[h].nbr for o in one]))
        assert np.array_equal(whole[h].eid, np.concatenate([o[h].eid for o in one]))
