"""tgl_sample_noalloc (workspace in the library's static device area) against
tgl_sample (caller's workspace), bit for bit, through the C ABI: two calls in
a row on the same GPU, the second with fewer roots, for several sampler
shapes; and the host-side rejection of a call whose workspace exceeds the
area."""
import ctypes as C
import math

import numpy as np
import pytest

import paper_2203_14883_amd as P
from paper_2203_14883_amd import binding as B
from paper_2203_14883_amd import workloads as W
from checks import assert_hops_equal
from gpu_util import announce, hops_to_numpy, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    return require_gpu()


def _noalloc(smp, g, roots, rts, mode, delta, seed, base):
    view = g.c_view()
    return P.lib().tgl_sample_noalloc(C.byref(view), roots.data_ptr(), rts.data_ptr(), roots.numel(),
                                      len(smp.fanouts), smp._fp, B.MODES[mode], smp.snapshots,
                                      C.c_float(delta), C.c_uint64(seed), C.c_uint64(base), smp._outs,
                                      smp.counts.data_ptr(), B._stream(None))


@pytest.mark.parametrize("fan,mode,S,delta", [((10, 10), "uniform", 1, math.inf),
                                              ((10, 10), "uniform", 3, 2.0e5),
                                              ((5, 3, 2), "recent", 1, math.inf)])
def test_noalloc_matches_workspace_call(torch, fan, mode, S, delta):
    w = W.make_c2()
    dev = torch.device("cuda")
    g = P.tcsr_build(*[torch.from_numpy(a).to(dev) for a in (w.src, w.dst, w.ts)], None, w.num_nodes, True)
    for b0, b1 in ((20, 140), (150, 160)):                  # the second call is smaller
        roots, rts, base = w.batches(b0, b1)
        r, t = torch.from_numpy(roots).to(dev), torch.from_numpy(rts).to(dev)
        announce("noalloc c2 batches %d..%d fan %s %s S=%d" % (b0, b1, fan, mode, S))
        ref = P.Sampler(len(roots), fan, S, device=dev)
        ref.run(g, r, t, mode, delta, 11, base)
        out = P.Sampler(len(roots), fan, S, device=dev)
        assert _noalloc(out, g, r, t, mode, delta, 11, base) == B.OK
        torch.cuda.synchronize()
        want, got = hops_to_numpy(ref.hops()), hops_to_numpy(out.hops())
        assert_hops_equal(got, want, "noalloc batches %d..%d" % (b0, b1))
        for h in range(len(fan)):
            assert got[h]["num_roots"] == want[h]["num_roots"]


def test_noalloc_rejects_oversized_call(torch):
    """A call whose workspace would not fit the static area is refused on the
    host: nothing is enqueued, the outputs keep their contents."""
    fan = (1024, 1024)
    n = 20000
    need = P.lib().tgl_sample_workspace(n, 2, B._i32_array(fan)[1], 1)
    assert need > B.NOALLOC_SCRATCH_BYTES
    dev = torch.device("cuda")
    w = W.make_c1()
    g = P.tcsr_build(*[torch.from_numpy(a).to(dev) for a in (w.src, w.dst, w.ts)], None, w.num_nodes, True)
    smp = P.Sampler(1, fan, 1, device=dev)
    smp.counts.fill_(-7)
    r = torch.zeros(n, dtype=torch.int32, device=dev)
    t = torch.zeros(n, dtype=torch.float32, device=dev)
    assert _noalloc(smp, g, r, t, "uniform", math.inf, 0, 0) == B.ENOSPACE
    torch.cuda.synchronize()
    assert smp.counts.cpu().tolist() == [-7, -7]
