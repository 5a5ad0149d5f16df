"""GPU path against the oracle over the whole argument range the C ABI
accepts, and with root counts whose grids exceed what the device holds at
once.

* 5-8 hops (up to TGL_MAX_HOPS) and fanouts 71-1024 (up to TGL_MAX_FANOUT),
  with and without snapshots, both modes, on dense random graphs.
* 3- and 4-hop sampling of a reduced c4 and of every c2 batch at once: the
  grid of every hop after the first is far larger than the resident blocks,
  so later wavefronts of a launch run after earlier ones have finished.  The
  per-group counts a hop writes and the offsets it reads from the previous
  hop must then live in different buffers.
* One run of more than half a billion entries, whose time directory has
  more cells than float32 counts exactly.
"""
import math

import numpy as np
import pytest

import oracle
import paper_2203_14883_amd as P
from paper_2203_14883_amd import workloads as W
from checks import assert_hops_equal
from gpu_util import announce, hops_to_numpy, require_gpu, upload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    return require_gpu()


def gpu_sample(g, roots, rts, fan, mode, S, D, seed, base):
    out = P.sample(g, upload(roots, np.int32), upload(rts, np.float32), fan, mode, S, D, seed, base)
    return hops_to_numpy(out)


def _dense_case(rng, trial):
    N = int(rng.integers(2, 40))
    m0 = int(rng.integers(100, 3000))
    src = rng.integers(0, N, m0).astype(np.int32)
    dst = rng.integers(0, N, m0).astype(np.int32)
    ts = rng.integers(0, 60, m0).astype(np.float32)
    und = bool(rng.integers(0, 4))
    eid = None if rng.integers(0, 2) else rng.integers(0, 10**12, m0).astype(np.int64)
    mode = ["recent", "uniform"][trial % 4 // 2]
    if trial % 2 == 0:
        hops = int(rng.integers(5, 9))
        fan = [int(rng.choice([1, 2, 3])) for _ in range(hops)]
        R = int(rng.integers(1, 300))
        S, D = [(1, math.inf), (2, 20.0), (3, 7.5), (9, 4.0)][int(rng.integers(0, 4))]
    else:
        fan = [int(rng.choice([71, 100, 255, 256, 513, 1000, 1024]))]
        fan += [int(rng.choice([1, 3, 71, 1024])) for _ in range(int(rng.integers(0, 2)))]
        R = int(rng.integers(1, 60 if len(fan) > 1 else 400))
        S, D = [(1, math.inf), (2, 11.0), (5, 6.0), (12, 3.0)][int(rng.integers(0, 4))]
        if len(fan) > 1 and fan[1] > 3:
            S, R = 1, min(R, 8)
    roots = rng.integers(0, N, R).astype(np.int32)
    rts = rng.integers(20, 62, R).astype(np.float32)
    return N, src, dst, ts, eid, und, roots, rts, fan, mode, S, D, int(rng.integers(0, 2**63)), int(rng.integers(0, 2**62))


def test_deep_hops_and_wide_fanouts(torch):
    """5-8 hops and fanouts above 70, up to 1024, on dense random graphs with
    1-12 snapshots (the wide first-hop kernel beyond 8)."""
    rng = np.random.default_rng(2025)
    deep = wide = 0
    for trial in range(60):
        N, src, dst, ts, eid, und, roots, rts, fan, mode, S, D, seed, base = _dense_case(rng, trial)
        announce("range trial %d N=%d m0=%d R=%d fan=%s mode=%s S=%d D=%s" % (trial, N, len(src), len(roots), fan,
                                                                             mode, S, D))
        og = oracle.build_tcsr(src, dst, ts, eid, N, und)
        g = P.tcsr_build(upload(src, np.int32), upload(dst, np.int32), upload(ts, np.float32),
                         None if eid is None else upload(eid, np.int64), N, und)
        want = oracle.sample(og, roots, rts, fan, mode, S, D, seed, base)
        got = gpu_sample(g, roots, rts, fan, mode, S, D, seed, base)
        assert_hops_equal(got, want, "range trial %d fan %s" % (trial, fan))
        for h in range(len(fan)):
            assert got[h]["num_roots"] == want[h].num_roots
        deep += len(fan) >= 5 and int((want[-1].nbr >= 0).sum()) > 0
        wide += fan[0] > 70 and int((want[0].nbr >= 0).sum()) > fan[0]
    assert deep >= 15 and wide >= 15, (deep, wide)


@pytest.fixture(scope="module")
def reduced_c4():
    w = W.make_c4(num_nodes=1_000_000, num_edges=10_700_000)
    og = oracle.build_tcsr(w.src, w.dst, w.ts, None, w.num_nodes, True)
    return w, og


@pytest.mark.parametrize("fan,mode", [((10, 10, 2), "uniform"), ((10, 10, 2), "recent"),
                                      ((10, 5, 2, 2), "uniform"), ((5, 3, 2, 2), "recent")])
def test_many_roots_multi_hop(torch, reduced_c4, fan, mode):
    """3 and 4 hops over 204,000 roots of a reduced c4 (17 batches): hops 2-4
    launch thousands of blocks, far beyond the resident ones."""
    w, og = reduced_c4
    g = P.tcsr_from_host(og.indptr, og.nbr, og.ts, og.eid)
    roots, rts, base = w.batches(1000, 1017)
    announce("reduced c4, %d roots, fan %s %s" % (len(roots), fan, mode))
    want = oracle.sample(og, roots, rts, fan, mode, 1, math.inf, 17, base)
    got = gpu_sample(g, roots, rts, fan, mode, 1, math.inf, 17, base)
    assert want[1].num_roots > 400_000, want[1].num_roots
    assert_hops_equal(got, want, "reduced c4 fan %s %s" % (fan, mode))
    for h in range(len(fan)):
        assert got[h]["num_roots"] == want[h].num_roots


@pytest.mark.parametrize("fan,mode,S,D", [((3, 2, 2, 2, 2), "uniform", 1, math.inf),
                                          ((2, 1, 2, 1, 2, 1, 2, 1), "recent", 1, math.inf),
                                          ((4, 2, 2), "uniform", 3, 2.0e5)])
def test_whole_c2_epoch_deep(torch, fan, mode, S, D):
    """Every c2 batch in one call (472,422 roots), 3-8 hops."""
    w = W.make_c2()
    og = oracle.build_tcsr(w.src, w.dst, w.ts, None, w.num_nodes, True)
    g = P.tcsr_from_host(og.indptr, og.nbr, og.ts, og.eid)
    roots, rts, base = w.batches(0, w.num_batches())
    announce("c2 epoch, %d roots, fan %s %s S=%d" % (len(roots), fan, mode, S))
    want = oracle.sample(og, roots, rts, fan, mode, S, D, 3, base)
    got = gpu_sample(g, roots, rts, fan, mode, S, D, 3, base)
    assert_hops_equal(got, want, "c2 epoch fan %s %s S=%d" % (fan, mode, S))
    for h in range(len(fan)):
        assert got[h]["num_roots"] == want[h].num_roots


def test_run_of_half_a_billion_entries(torch):
    """One run of 2^29 + 2^20 entries (integer timestamps below 1e7, so heavy
    ties), whose time directory has 2^24 + 2^15 cells: more than float32
    holds integers exactly, so the cell count is rounded where the build and
    the sampler place times in cells, and they must still agree.  The
    directory is checked slot by slot against its definition; 100,000 roots
    on the run (and on an empty one), sampled in three snapshots in both
    modes, are compared with the oracle on the same T-CSR copied to the host."""
    from gpu_util import check_dir_slots
    L = (1 << 29) + (1 << 20)
    dev = torch.device("cuda")
    gen = torch.Generator(device=dev)
    gen.manual_seed(2029)
    announce("half-a-billion run: build of %d entries" % L)
    src = torch.zeros(L, dtype=torch.int32, device=dev)
    dst = torch.ones(L, dtype=torch.int32, device=dev)
    ts = torch.randint(0, 10_000_000, (L,), device=dev, generator=gen, dtype=torch.int32).float()
    g = P.tcsr_build(src, dst, ts, None, 2, undirected=False, hist=False, dir=True)
    del src, dst
    assert g.indptr.tolist() == [0, L, L]
    assert bool((g.ts[1:] >= g.ts[:-1]).all()), "the run is not sorted by time"
    want_sorted, _ = torch.sort(ts)
    assert torch.equal(g.ts, want_sorted), "the run's timestamps differ from the input's"
    del ts, want_sorted
    torch.cuda.empty_cache()
    K = -(-L // 32)
    assert K > (1 << 24)
    announce("half-a-billion run: directory of %d cells" % K)
    check_dir_slots(g)
    announce("half-a-billion run: host copy")
    tsh = g.ts.cpu().numpy()
    og = oracle.TCSR(np.array([0, L, L], np.int64), np.ones(L, np.int32), g.entries[:, 1].contiguous().cpu().numpy(), tsh)
    rng = np.random.default_rng(2029)
    R = 100_000
    roots = np.where(rng.random(R) < 0.95, 0, rng.integers(1, 3, R)).astype(np.int32)   # 2: outside the graph
    rts = rng.uniform(-1e6, 1.1e7, R).astype(np.float32)
    rts[: R // 4] = tsh[rng.integers(0, L, R // 4)]                                      # on timestamps
    for mode in ("recent", "uniform"):
        announce("half-a-billion run: %s" % mode)
        want = oracle.sample(og, roots, rts, [10], mode, 3, 1e5, 7, 11)
        got = gpu_sample(g, roots, rts, [10], mode, 3, 1e5, 7, 11)
        assert_hops_equal(got, want, "half-a-billion run, %s" % mode)
        assert int((want[0].nbr >= 0).sum()) > R
    del g, og
    torch.cuda.empty_cache()
