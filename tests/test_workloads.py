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
