"""Seeded synthetic temporal-graph workloads.

This module only draws random inputs: an edge list (COO) with timestamps and
edge ids, and chronological streams of root queries.  It holds none of the
sampler's arithmetic (no sorting into T-CSR, no window location, no neighbour
selection), so both the CPU oracle and the GPU path can be fed from it.

The five presets copy the shapes the paper evaluates on, since the datasets
themselves are not available (Table 3, Section 4.1):

* ``c1`` tiny bipartite graph, 1-hop most-recent sampling (TGN-style, Sec. 4.2)
* ``c2`` Wikipedia-shaped bipartite graph (Table 3), 2-hop uniform 10x10
  (TGAT-style, Sec. 4.2), batches of 600 edges + 1 negative per edge
* ``c3`` GDELT-shaped dense long-history graph (Table 3, Sec. 4.1.1),
  1-hop most-recent inside 3 dynamic snapshots
* ``c4`` MAG-shaped billion-edge citation graph (Table 3, Sec. 4.1.2),
  timestamps are publication years, 2-hop uniform 10x10
* ``c5`` 100M-edge power-law graph, 2-hop uniform inside 3 snapshots, with
  the build input given as an unsorted (shuffled) COO

Every array is a deterministic function of the preset's seed: generation is
split into fixed-size chunks, each with its own ``SeedSequence`` child, so the
result does not depend on how many threads run the chunks.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Callable, Optional, Sequence

import numpy as np

__all__ = ["Workload", "make", "PRESETS", "make_c1", "make_c2", "make_c3",
           "make_c4", "make_c5"]

_CHUNK = 1 << 24          # elements per independently seeded chunk
_NEG_TAG = 0x6E6567       # stream tag for negative destinations ("neg")
_CHUNK_TAG = 0x63686B     # stream tag for random chunk scheduling offsets ("chk")
_CNEG_TAG = 0x636E67      # stream tag for negatives of chunk-scheduled batches ("cng")


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _run_chunks(n: int, fn: Callable[[int, int, int], None], chunk: int = _CHUNK) -> None:
    """Call ``fn(index, begin, end)`` for fixed chunks of ``range(n)``."""
    nch = (n + chunk - 1) // chunk
    if nch <= 1:
        if n:
            fn(0, 0, n)
        return
    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(lambda c: fn(c, c * chunk, min(n, (c + 1) * chunk)), range(nch)))


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def _zipf_cdf(n: int, s: float) -> np.ndarray:
    """CDF of the finite Zipf law P(rank r) ~ r^-s over ranks 1..n."""
    w = np.arange(1, n + 1, dtype=np.float64) ** (-float(s))
    c = np.cumsum(w)
    c /= c[-1]
    return c


def _zipf_ids(seed: int, tag: int, cdf: np.ndarray, rank_to_id: np.ndarray,
              size: int, offset: int = 0) -> np.ndarray:
    """``size`` Zipf-distributed node ids (inverse CDF, ranks mapped through a permutation)."""
    out = np.empty(size, dtype=np.int32)
    last = len(cdf) - 1

    def fill(c: int, b: int, e: int) -> None:
        u = _rng(seed, tag, c).random(e - b)
        r = np.searchsorted(cdf, u, side="right")
        np.minimum(r, last, out=r)
        out[b:e] = rank_to_id[r] + offset

    _run_chunks(size, fill)
    return out


def _sorted_uniform_f32(seed: int, tag: int, n: int, hi: float) -> np.ndarray:
    """n sorted draws of U[0, hi), via normalised exponential spacings, rounded to float32."""
    e = _rng(seed, tag).standard_exponential(n + 1)
    c = np.cumsum(e)
    t = c[:n] * (hi / c[n])
    return t.astype(np.float32)


@dataclass
class Workload:
    """A temporal graph plus the sampler settings and root stream of one preset.

    Edges are listed chronologically (``ts`` non-decreasing).  ``eid is None``
    means edge ids equal edge positions.  ``build_order`` (optional) is the
    permutation in which the COO is handed to the T-CSR build; ``None`` means
    chronological order.
    """
    name: str
    num_nodes: int
    src: np.ndarray
    dst: np.ndarray
    ts: np.ndarray
    eid: Optional[np.ndarray]
    undirected: bool
    hops: int
    fanouts: tuple
    mode: str                    # "recent" or "uniform"
    snapshots: int
    snapshot_len: float          # math.inf when there is a single unbounded window
    sample_seed: int
    batch_edges: int
    negatives: bool              # roots = [src; dst; neg] (True) or [src; dst]
    neg_range: tuple = (0, 0)    # negative destinations drawn uniformly from [lo, hi)
    gen_seed: int = 0
    default_batches: Optional[Sequence[int]] = None
    build_order: Optional[np.ndarray] = None
    meta: dict = field(default_factory=dict)

    @property
    def num_edges(self) -> int:
        return int(self.src.shape[0])

    @property
    def roots_per_edge(self) -> int:
        return 3 if self.negatives else 2

    def num_batches(self) -> int:
        return (self.num_edges + self.batch_edges - 1) // self.batch_edges

    def edge_ids(self) -> np.ndarray:
        return np.arange(self.num_edges, dtype=np.int64) if self.eid is None else self.eid

    def root_base(self, b: int) -> int:
        """Global index of the first root of batch ``b`` (all earlier batches are full)."""
        return b * self.batch_edges * self.roots_per_edge

    def negatives_of(self, b: int) -> np.ndarray:
        e0 = b * self.batch_edges
        e1 = min(self.num_edges, e0 + self.batch_edges)
        lo, hi = self.neg_range
        return _rng(self.gen_seed, _NEG_TAG, b).integers(lo, hi, size=e1 - e0).astype(np.int32)

    def batch(self, b: int):
        """Roots of batch ``b``: (node ids int32, query times float32, root_base)."""
        if not 0 <= b < self.num_batches():
            raise IndexError(b)
        e0 = b * self.batch_edges
        e1 = min(self.num_edges, e0 + self.batch_edges)
        parts = [self.src[e0:e1], self.dst[e0:e1]]
        if self.negatives:
            parts.append(self.negatives_of(b))
        t = self.ts[e0:e1]
        roots = np.concatenate(parts).astype(np.int32, copy=False)
        root_ts = np.concatenate([t] * len(parts)).astype(np.float32, copy=False)
        return roots, root_ts, self.root_base(b)

    def chunk_schedule(self, epoch: int, chunk_edges: int, batch_edges: Optional[int] = None):
        """Random chunk scheduling (Alg. 2): the training edges are cut into
        chunks of ``chunk_edges``; each epoch starts its batches of
        ``batch_edges`` (default: the preset's) at a randomly chosen chunk
        boundary inside the first batch, and keeps only whole batches, so that
        neighbouring chunks fall into different mini-batches from one epoch to
        the next.  Returns the epoch's batches as edge ranges ``(e_s, e_e)``.

        The printed start offset is rand(0, bs/cs) * bs, a whole number of
        batches, which would not move any chunk relative to the batch grid;
        following the text (one chunk picked as the starting point) the
        offset is read as rand(0, bs/cs) * cs."""
        bs = int(batch_edges or self.batch_edges)
        cs = int(chunk_edges)
        if cs < 1 or bs % cs != 0:
            raise ValueError("the chunk size must divide the batch size")
        e_s = int(_rng(self.gen_seed, _CHUNK_TAG, int(epoch)).integers(0, bs // cs)) * cs
        out = []
        while e_s + bs <= self.num_edges:
            out.append((e_s, e_s + bs))
            e_s += bs
        return out

    def edge_batch(self, e0: int, e1: int, epoch: int = 0):
        """Roots of the edges [e0, e1) -- sources, destinations and (if the
        preset has them) one uniform negative destination per edge, drawn from
        a stream keyed by (epoch, e0) -- with root_base = roots_per_edge * e0,
        so that the batches of one epoch have disjoint root indices whatever
        their offsets."""
        if not 0 <= e0 <= e1 <= self.num_edges:
            raise IndexError((e0, e1))
        parts = [self.src[e0:e1], self.dst[e0:e1]]
        if self.negatives:
            lo, hi = self.neg_range
            parts.append(_rng(self.gen_seed, _CNEG_TAG, int(epoch), int(e0)).integers(lo, hi, size=e1 - e0)
                         .astype(np.int32))
        t = self.ts[e0:e1]
        roots = np.concatenate(parts).astype(np.int32, copy=False)
        root_ts = np.concatenate([t] * len(parts)).astype(np.float32, copy=False)
        return roots, root_ts, self.roots_per_edge * e0

    def batches(self, b0: int, b1: int):
        """Concatenated roots of batches [b0, b1): consecutive root_base ranges."""
        rs, ts = [], []
        for b in range(b0, b1):
            r, t, _ = self.batch(b)
            rs.append(r)
            ts.append(t)
        return np.concatenate(rs), np.concatenate(ts), self.root_base(b0)

    def build_input(self):
        """(src, dst, ts, eid-or-None) in the order the T-CSR build receives them."""
        if self.build_order is None:
            return self.src, self.dst, self.ts, self.eid
        p = self.build_order
        eid = p.astype(np.int64) if self.eid is None else self.eid[p]
        return self.src[p], self.dst[p], self.ts[p], eid

    def sampler_args(self) -> dict:
        return dict(fanouts=tuple(self.fanouts), mode=self.mode,
                    snapshots=self.snapshots, snapshot_len=self.snapshot_len,
                    seed=self.sample_seed)


# --------------------------------------------------------------------------
# presets
# --------------------------------------------------------------------------

def make_c1(n_side: int = 1000, num_edges: int = 20_000, seed: int = 0) -> Workload:
    """Tiny bipartite graph: src ids [0, n), dst ids [n, 2n), Zipf(1.2) per side,
    integer-valued timestamps uniform in [0, 1e6), 1-hop most-recent k=10 for the
    200 endpoints of the last 100 edges."""
    cdf = _zipf_cdf(n_side, 1.2)
    rng = _rng(seed, 1)
    p_src = rng.permutation(n_side).astype(np.int32)
    p_dst = rng.permutation(n_side).astype(np.int32)
    src = _zipf_ids(seed, 2, cdf, p_src, num_edges)
    dst = _zipf_ids(seed, 3, cdf, p_dst, num_edges, offset=n_side)
    ts = np.sort(_rng(seed, 4).integers(0, 1_000_000, size=num_edges)).astype(np.float32)
    nb = (num_edges + 99) // 100
    return Workload("c1", 2 * n_side, src, dst, ts, None, True, 1, (10,), "recent",
                    1, math.inf, seed, 100, False, gen_seed=seed,
                    default_batches=[nb - 1])


def make_c2(n_users: int = 8227, n_items: int = 1000, num_edges: int = 157_474,
            seed: int = 1) -> Workload:
    """Wikipedia-shaped bipartite interactions: users Zipf(1.1), items Zipf(1.3),
    timestamps uniform over [0, 2.7e6) s; batches of 600 edges with one uniform
    negative item per edge; 2-hop uniform 10x10."""
    rng = _rng(seed, 1)
    p_u = rng.permutation(n_users).astype(np.int32)
    p_i = rng.permutation(n_items).astype(np.int32)
    src = _zipf_ids(seed, 2, _zipf_cdf(n_users, 1.1), p_u, num_edges)
    dst = _zipf_ids(seed, 3, _zipf_cdf(n_items, 1.3), p_i, num_edges, offset=n_users)
    ts = _sorted_uniform_f32(seed, 4, num_edges, 2.7e6)
    return Workload("c2", n_users + n_items, src, dst, ts, None, True, 2, (10, 10),
                    "uniform", 1, math.inf, seed, 600, True,
                    neg_range=(n_users, n_users + n_items), gen_seed=seed)


def make_c3(num_nodes: int = 16_682, num_edges: int = 191_000_000,
            t_buckets: int = 170_000, seed: int = 2) -> Workload:
    """GDELT-shaped graph: both endpoints Zipf(1.05) over one popularity ranking,
    integer timestamps (15-minute buckets) uniform over [0, t_buckets) with heavy
    ties; batches of 4,000 edges x 3 roots; 1-hop most-recent k=10 in each of 3
    snapshot windows of length 1e4."""
    cdf = _zipf_cdf(num_nodes, 1.05)
    perm = _rng(seed, 1).permutation(num_nodes).astype(np.int32)
    src = _zipf_ids(seed, 2, cdf, perm, num_edges)
    dst = _zipf_ids(seed, 3, cdf, perm, num_edges)
    counts = _rng(seed, 4).multinomial(num_edges, np.full(t_buckets, 1.0 / t_buckets))
    ts = np.repeat(np.arange(t_buckets, dtype=np.float32), counts)
    return Workload("c3", num_nodes, src, dst, ts, None, True, 1, (10,), "recent",
                    3, 1.0e4, seed, 4000, True, neg_range=(0, num_nodes), gen_seed=seed)


def make_c4(num_nodes: int = 121_700_000, num_edges: int = 1_300_000_000,
            alpha: float = 2.1, max_deg: int = 100_000, year0: int = 1900,
            year1: int = 2021, growth: float = 1.04, seed: int = 3) -> Workload:
    """MAG-shaped citation graph.  Each node (paper) gets a publication year with
    P(y) ~ growth^(y - year0) on [year0, year1); an out-degree drawn as
    floor(x) with x classical-Pareto(alpha) scaled to the target mean, capped at
    ``max_deg`` and rescaled so the degrees sum to exactly ``num_edges``.  An
    edge u->v has the citing paper's year as timestamp and v uniform among the
    papers of year <= year(u).  Edges are listed year by year (random paper
    order inside a year).  Batches of 4,000 edges x 3 roots; 2-hop uniform 10x10."""
    n = int(num_nodes)
    years = np.arange(year0, year1)
    py = growth ** (years - year0).astype(np.float64)
    ycdf = np.cumsum(py)
    ycdf /= ycdf[-1]
    ny = len(years)

    year_of = np.empty(n, dtype=np.int16)

    def f_year(c, b, e):
        r = np.searchsorted(ycdf, _rng(seed, 1, c).random(e - b), side="right")
        np.minimum(r, ny - 1, out=r)
        year_of[b:e] = r

    _run_chunks(n, f_year)

    mean = num_edges / n
    xm = mean * (alpha - 1.0) / alpha
    deg = np.empty(n, dtype=np.int64)

    def f_deg(c, b, e):
        x = xm * (1.0 + _rng(seed, 2, c).pareto(alpha, e - b))
        deg[b:e] = np.minimum(np.floor(x), max_deg).astype(np.int64)

    _run_chunks(n, f_deg)
    tot = int(deg.sum())
    deg = (deg * num_edges) // tot                  # floor(d * E / T), sum <= E
    short = int(num_edges - deg.sum())              # 0 <= short < n
    if short:
        bump = _rng(seed, 3).permutation(n)[:short]
        deg[bump] += 1
    assert int(deg.sum()) == num_edges

    # paper order: sorted by year, random order within a year
    perm = _rng(seed, 4).permutation(n)
    node_seq = perm[np.argsort(year_of[perm], kind="stable")].astype(np.int32)
    del perm
    deg_seq = deg[node_seq]
    nodes_per_year = np.bincount(year_of, minlength=ny).astype(np.int64)
    cum_nodes = np.cumsum(nodes_per_year)                        # papers with year <= y
    node_off = np.concatenate([[0], cum_nodes])
    edge_off_nodes = np.concatenate([[0], np.cumsum(deg_seq)])   # edge offset of each node_seq entry

    src = np.empty(num_edges, dtype=np.int32)
    dst = np.empty(num_edges, dtype=np.int32)
    ts = np.empty(num_edges, dtype=np.float32)

    # src: repeat node_seq by degree (chunks over nodes)
    def f_src(c, b, e):
        s0, s1 = edge_off_nodes[b], edge_off_nodes[e]
        src[s0:s1] = np.repeat(node_seq[b:e], deg_seq[b:e])

    _run_chunks(n, f_src, chunk=1 << 22)

    tasks = []
    for y in range(ny):
        e0 = int(edge_off_nodes[node_off[y]])
        e1 = int(edge_off_nodes[node_off[y + 1]])
        ts[e0:e1] = np.float32(year0 + y)
        for c, b in enumerate(range(e0, e1, _CHUNK)):
            tasks.append((y, c, b, min(e1, b + _CHUNK)))

    def f_dst(task):
        y, c, b, e = task
        cy = int(cum_nodes[y])
        idx = (_rng(seed, 5, y, c).random(e - b) * cy).astype(np.int64)
        np.minimum(idx, cy - 1, out=idx)
        dst[b:e] = node_seq[idx]

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(f_dst, tasks))

    return Workload("c4", n, src, dst, ts, None, True, 2, (10, 10), "uniform",
                    1, math.inf, seed, 4000, True, neg_range=(0, n), gen_seed=seed,
                    meta=dict(max_deg=max_deg, alpha=alpha))


def make_c5(num_nodes: int = 10_000_000, num_edges: int = 100_000_000,
            t_max: float = 1.0e8, batch_edges: int = 60_000, seed: int = 4) -> Workload:
    """Power-law graph: both endpoints Zipf(1.2) over one ranking, float32
    timestamps uniform in [0, 1e8); the T-CSR build receives the COO in a seeded
    random order; batches of 60,000 edges x 3 roots; 2-hop uniform 10x10 inside 3
    snapshot windows of length 1e6."""
    cdf = _zipf_cdf(num_nodes, 1.2)
    perm = _rng(seed, 1).permutation(num_nodes).astype(np.int32)
    src = _zipf_ids(seed, 2, cdf, perm, num_edges)
    dst = _zipf_ids(seed, 3, cdf, perm, num_edges)
    ts = _sorted_uniform_f32(seed, 4, num_edges, t_max)
    order = _rng(seed, 5).permutation(num_edges).astype(np.int64)
    return Workload("c5", num_nodes, src, dst, ts, None, True, 2, (10, 10), "uniform",
                    3, 1.0e6, seed, batch_edges, True, neg_range=(0, num_nodes),
                    gen_seed=seed, build_order=order)


PRESETS = {"c1": make_c1, "c2": make_c2, "c3": make_c3, "c4": make_c4, "c5": make_c5}


def make(name: str, **kw) -> Workload:
    return PRESETS[name](**kw)
