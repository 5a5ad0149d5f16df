"""tgl_mfg_export (through the C ABI) against the MFG block oracle, byte for
byte: blocks of every hop of GPU sampling calls on a Wikipedia-shaped graph
(uniform and most-recent, one and several windows, three hops), a call with
no roots and one whose slots are all PAD."""
import math

import numpy as np
import pytest

import oracle
from oracle import mfg as M
import paper_2203_14883_amd as P
from paper_2203_14883_amd import workloads as W
from gpu_util import announce, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    return require_gpu()


def _compare(got, want, what):
    s = got.sliced()
    G, E = (int(v) for v in s.sizes.cpu().tolist())
    assert (G, E) == (want["G"], want["E"]), what + ": sizes"
    for f in ("indptr", "edge_dst", "edge_eid", "edge_dt", "src_nid", "src_ts"):
        a = getattr(s, f).cpu().numpy()
        assert a.dtype == want[f].dtype and a.tobytes() == want[f].tobytes(), "%s: %s differs" % (what, f)


def test_blocks_of_sampled_hops(torch):
    w = W.make_c2(n_users=2000, n_items=300, num_edges=40_000, seed=23)
    og = oracle.build_tcsr(w.src, w.dst, w.ts, None, w.num_nodes, True)
    g = P.tcsr_from_host(og.indptr, og.nbr, og.ts, og.eid)
    roots, rts, base = w.batches(4, 10)
    d_r, d_t = torch.from_numpy(roots).cuda(), torch.from_numpy(rts).cuda()
    for fan, mode, S, D in [((10, 10), "uniform", 1, math.inf), ((10, 5), "recent", 1, math.inf),
                            ((6, 4), "recent", 3, 3.0e4), ((5, 3, 2), "uniform", 2, 6.0e4)]:
        announce("mfg blocks fan=%s mode=%s S=%d" % (fan, mode, S))
        smp = P.Sampler(len(roots), fan, S)
        smp.run(g, d_r, d_t, mode, D, 9, base)
        want_hops = oracle.sample(og, roots, rts, fan, mode, S, D, 9, base)
        for h, k in enumerate(fan):
            blk = P.mfg_export(smp, h, d_r, d_t)
            want = M.block(want_hops[h], want_hops[h - 1] if h else None, roots, rts, S if h == 0 else 1, k)
            _compare(blk, want, "fan=%s S=%d hop %d" % (fan, S, h + 1))


def test_degenerate_blocks(torch):
    w = W.make_c2(n_users=300, n_items=40, num_edges=3000, seed=2)
    og = oracle.build_tcsr(w.src, w.dst, w.ts, None, w.num_nodes, True)
    g = P.tcsr_from_host(og.indptr, og.nbr, og.ts, og.eid)
    announce("mfg with no roots")
    smp = P.Sampler(8, (4, 4), 1)
    e_r = torch.zeros(0, dtype=torch.int32, device="cuda")
    e_t = torch.zeros(0, dtype=torch.float32, device="cuda")
    smp.run(g, e_r, e_t, "uniform", math.inf, 1, 0)
    for h in range(2):
        s = P.mfg_export(smp, h, e_r, e_t).sliced()
        assert s.sizes.cpu().tolist() == [0, 0] and s.indptr.cpu().tolist() == [0]
    announce("mfg with all slots PAD")
    roots = np.array([0, 1, 2], np.int32)
    rts = np.full(3, -1.0, np.float32)              # before every edge: no candidates
    d_r, d_t = torch.from_numpy(roots).cuda(), torch.from_numpy(rts).cuda()
    smp = P.Sampler(3, (4, 4), 1)
    smp.run(g, d_r, d_t, "uniform", math.inf, 1, 0)
    s = P.mfg_export(smp, 0, d_r, d_t).sliced()
    assert s.sizes.cpu().tolist() == [3, 0] and s.indptr.cpu().tolist() == [0, 0, 0, 0]
    assert s.src_nid.cpu().tolist() == [0, 1, 2]
