"""The oracle against the hand-worked example of tests/golden/fig3_tcsr.txt
(structure of the paper's Figure 3, Section 3.1; values derived by hand)."""
import math

import numpy as np
import pytest

import oracle
from golden_io import floats, ints, read

G = read("fig3_tcsr.txt")


def _graph(undirected):
    return oracle.build_tcsr(ints(G["coo_src"]), ints(G["coo_dst"]), floats(G["coo_ts"]),
                             ints(G["coo_eid"]), int(G["num_nodes"][0]), undirected)


@pytest.mark.parametrize("kind", ["directed", "undirected"])
def test_build(kind):
    g = _graph(kind == "undirected")
    assert np.array_equal(g.indptr, ints(G[kind + ".indptr"]))
    assert np.array_equal(g.nbr, ints(G[kind + ".nbr"]))
    assert np.array_equal(g.eid, ints(G[kind + ".eid"]))
    assert np.array_equal(g.ts, floats(G[kind + ".ts"]).astype(np.float32))


def _slots(rows):
    a = np.array(rows, dtype=np.float64).reshape(-1, 4)
    return (a[:, 0].astype(np.int32), a[:, 1].astype(np.int64),
            a[:, 2].astype(np.float32), a[:, 3].astype(np.float32))


@pytest.mark.parametrize("q", ["D1", "U1", "U2"])
def test_query(q):
    g = _graph(G[q + ".graph"][0] == "undirected")
    S = int(G[q + ".snapshots"][0])
    delta = math.inf if G[q + ".snapshots"][1] == "inf" else float(G[q + ".snapshots"][1])
    fan = [int(k) for k in G[q + ".fanouts"]]
    out = oracle.sample(g, ints(G[q + ".roots"]), floats(G[q + ".root_ts"]), fan, "recent",
                        S, delta, seed=0, root_base=0)
    for h in range(len(fan)):
        nbr, eid, ts, dt = _slots(G["%s.hop%d.slots" % (q, h + 1)])
        o = out[h]
        assert np.array_equal(o.nbr, nbr), (h, o.nbr, nbr)
        assert np.array_equal(o.eid, eid)
        assert np.array_equal(o.ts.view(np.uint32), ts.view(np.uint32))
        assert np.array_equal(o.dt.view(np.uint32), dt.view(np.uint32))
        if h > 0:
            assert np.array_equal(o.parent, ints(G["%s.hop%d.parent" % (q, h + 1)]))
