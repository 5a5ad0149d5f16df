"""GPU path against the oracle at the full preset sizes, in the launch
configuration bench.py times.

* c4 (121.7M nodes, 1.3B edges, 2.6B T-CSR entries): two whole benchmark
  steps (64 batches, 768,000 roots, 2 hops) are compared slot for slot with
  the oracle, which builds the full runs of every node the step reaches.
* c3 (191M edges, runs up to ~4.6e7 entries; 1 hop in 3 snapshots) and c5
  (200M entries built from a shuffled COO; 2 hops inside 3 snapshots): the
  whole GPU T-CSR is compared byte for byte with the oracle's build of the
  same COO (indptr, nbr, eid, ts; node records, search index and
  neighbour-first hints against their definitions), and two whole
  benchmark steps each (c3: 64 batches = 768,000 roots; c5: one batch =
  180,000 roots) slot for slot with the oracle on that T-CSR.
* For c4 the GPU T-CSR is checked in full on the device (indptr, degrees,
  sortedness of every run, the timestamp array, the hints) and the runs of
  sampled nodes bit for bit against the oracle's.
* Every full-size build's neighbour histories are checked on the device
  against their definition (the lower bound of each entry's time in its
  neighbour's run).  The c4 steps sample through them.
* Every full-size build's time directory is checked slot by slot: each
  cell's position is where its run's cells reach that cell, and its
  timestamp is that entry's.  The c3 and c5 steps search through them.
"""
import gc

import numpy as np
import pytest

import oracle
import paper_2203_14883_amd as P
from oracle import subgraph
from paper_2203_14883_amd import workloads as W
from checks import assert_hops_equal, same_bits
from gpu_util import announce, check_dir_slots, check_hist_device, hops_to_numpy, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    return require_gpu()


def build_on_gpu(torch, w):
    src, dst, ts, eid = w.build_input()
    dev = torch.device("cuda")
    d = [torch.from_numpy(a).to(dev) for a in (src, dst, ts)]
    de = None if eid is None else torch.from_numpy(eid).to(dev)
    g = P.tcsr_build(d[0], d[1], d[2], de, w.num_nodes, w.undirected)
    # device-side invariants of the whole structure
    M = g.num_entries
    ip = g.indptr
    assert int(ip[0]) == 0 and int(ip[-1]) == M and bool((ip[1:] >= ip[:-1]).all())
    deg = torch.bincount(d[0].long(), minlength=w.num_nodes)
    if w.undirected:
        deg += torch.bincount(d[1].long(), minlength=w.num_nodes)
    assert torch.equal(deg, ip[1:] - ip[:-1]), "degrees differ from the edge list"
    del d, de, deg
    start = torch.zeros(M, dtype=torch.bool, device=dev)
    start[ip[:-1][ip[:-1] < M]] = True
    ts_arr = g.ts
    bad = (ts_arr[1:] < ts_arr[:-1]) & ~start[1:]
    assert int(bad.sum()) == 0, "a run is not sorted by time"
    assert torch.equal(ts_arr.view(torch.int32), g.entries.view(torch.int32)[:, 1]), "ts array differs"
    del start, bad
    # neighbour-first hints of every entry against their definition (the
    # neighbour's first timestamp is not below the entry's), in chunks
    first = torch.full((w.num_nodes,), float("inf"), dtype=torch.float32, device=dev)
    ne = ip[1:] > ip[:-1]
    first[ne] = ts_arr[ip[:-1][ne]]
    words = g.entries.view(torch.int32)
    for c0 in range(0, M, 1 << 28):
        w0 = words[c0:c0 + (1 << 28), 0]
        want = ~(first[(w0 & 0x7FFFFFFF).long()] < ts_arr[c0:c0 + (1 << 28)])
        assert torch.equal(w0 < 0, want), "neighbour-first hints differ in entries %d.." % c0
    del first, ne, words
    torch.cuda.empty_cache()
    # neighbour histories of every entry against their definition
    check_hist_device(g)
    # time directory of every run, slot by slot
    check_dir_slots(g)
    return g


def torch_mod():
    import torch
    return torch


def check_runs(g, og, nodes):
    """GPU runs of ``nodes`` equal the oracle's runs bit for bit."""
    ip = g.indptr.cpu().numpy()
    for x in nodes:
        a, b = int(ip[x]), int(ip[x + 1])
        c, d = int(og.indptr[x]), int(og.indptr[x + 1])
        assert b - a == d - c, "run length of node %d" % x
        ent = g.entries[a:b].cpu().numpy()
        w4 = ent.view(np.int32).reshape(-1, 4)
        assert np.array_equal(w4[:, 0] & 0x7FFFFFFF, og.nbr[c:d]), "nbr of node %d" % x
        assert np.array_equal(ent[:, 1], og.eid[c:d]), "eid of node %d" % x
        assert same_bits(w4[:, 1].copy().view(np.float32), og.ts[c:d]), "ts of node %d" % x
        rec = g.nodes[x].cpu().numpy()
        bounds = rec[:2].view(np.uint32)
        assert bounds[0] == a and bounds[1] == b, "node record bounds of node %d" % x
        inl = np.full(28, np.inf, np.float32)
        inl[:min(28, d - c)] = og.ts[c:c + min(28, d - c)]
        first = og.ts[c] if d > c else np.float32(np.inf)
        last = og.ts[d - 1] if d > c else np.float32(-np.inf)
        assert same_bits(rec[2:4].copy().view(np.float32), np.array([first, last], np.float32)), \
            "node record first/last of node %d" % x
        assert same_bits(rec[4:].copy().view(np.float32), inl), "node record inline ts of node %d" % x
    if g.ts_index is not None and g.num_entries:
        j = np.unique(np.random.default_rng(5).integers(0, g.ts_index.numel(), 4096))
        jt = torch_mod().from_numpy(j).to(g.ts.device)
        assert same_bits(g.ts_index[jt].cpu().numpy(), g.ts[jt * 32].cpu().numpy()), "search index"


def gpu_step(torch, g, w, b0, B):
    roots, rts, base = w.batches(b0, b0 + B)
    smp = P.Sampler(len(roots), w.fanouts, w.snapshots)
    r, t = torch.from_numpy(roots).cuda(), torch.from_numpy(rts).cuda()
    smp.run(g, r, t, w.mode, w.snapshot_len, w.sample_seed, base)
    return roots, rts, base, hops_to_numpy(smp.hops())


def test_c4_full_step(torch):
    announce("c4 full size: generate")
    w = W.make_c4()
    announce("c4 full size: GPU build of %d edges" % w.num_edges)
    g = build_on_gpu(torch, w)
    B = 64
    for b0 in (0, w.num_batches() // 2):
        announce("c4 step at batch %d: GPU sample" % b0)
        roots, rts, base, got = gpu_step(torch, g, w, b0, B)
        announce("c4 step at batch %d: oracle on the reached sub-graph" % b0)
        src, dst, ts, eid = w.build_input()
        og = subgraph.reach_tcsr(src, dst, ts, eid, w.num_nodes, True, roots, rts, w.fanouts, w.mode,
                                 w.snapshots, w.snapshot_len, w.sample_seed, base)
        want = oracle.sample(og, roots, rts, w.fanouts, w.mode, w.snapshots, w.snapshot_len,
                             w.sample_seed, base)
        assert_hops_equal(got, want, "c4 step at batch %d" % b0)
        rng = np.random.default_rng(b0)
        check_runs(g, og, rng.choice(np.unique(roots), 300, replace=False))
    del g
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["c3", "c5"])
def test_full_size_whole_steps(torch, name):
    from gpu_util import tcsr_to_host
    from test_gpu_parity import assert_tcsr_equal
    announce("%s full size: generate" % name)
    w = W.make(name)
    announce("%s full size: GPU build of %d edges" % (name, w.num_edges))
    g = build_on_gpu(torch, w)
    announce("%s full size: oracle build of the same COO" % name)
    src, dst, ts, eid = w.build_input()
    og = oracle.build_tcsr(src, dst, ts, eid, w.num_nodes, w.undirected)
    del src, dst, ts, eid
    gc.collect()
    announce("%s full size: T-CSR byte for byte" % name)
    assert_tcsr_equal(tcsr_to_host(g, hist_on_host=False, dir_on_host=False), og, "%s full size" % name)
    gc.collect()
    B = 64 if name == "c3" else 1
    for b0 in (w.num_batches() // 2, w.num_batches() - B):
        announce("%s step at batch %d (%d batches): GPU sample" % (name, b0, B))
        roots, rts, base, got = gpu_step(torch, g, w, b0, B)
        announce("%s step at batch %d: oracle" % (name, b0))
        want = oracle.sample(og, roots, rts, w.fanouts, w.mode, w.snapshots, w.snapshot_len,
                             w.sample_seed, base)
        assert_hops_equal(got, want, "%s step at batch %d" % (name, b0))
        for h in range(len(w.fanouts)):
            assert got[h]["num_roots"] == want[h].num_roots
    del g
    gc.collect()
    torch.cuda.empty_cache()
