"""Pins of the MFG block oracle (oracle/mfg.py):

* the vectorised definition against explicit loops over groups and slots;
* properties the sampler's definition fixes: every edge goes from a source
  node strictly earlier than its destination (ts < t), with dt the float
  difference of the two times; a group's edges are its valid slots, newest
  first for most-recent sampling; the edge count is the number of valid
  slots; the destination nodes of hop 2 are the valid slots of hop 1;
* plausible mistakes (an inclusive scan, no destination prefix in the source
  arrays, edges attached to slots instead of groups, hop-1 destinations not
  repeated per window) each fail a check.
"""
import math

import numpy as np
import pytest

import oracle
from oracle import mfg as M
from paper_2203_14883_amd import workloads as W


def _case(mode, S, D):
    w = W.make_c2(n_users=500, n_items=60, num_edges=9000, seed=4)
    g = oracle.build_tcsr(w.src, w.dst, w.ts, None, w.num_nodes, True)
    roots, rts, base = w.batches(2, 6)
    hops = oracle.sample(g, roots, rts, (10, 4), mode, S, D, 3, base)
    return roots, rts, hops, S


CASES = [("uniform", 1, math.inf), ("recent", 1, math.inf), ("recent", 3, 3.0e4), ("uniform", 2, 5.0e4)]


def _checks(block):
    for mode, S, D in CASES:
        roots, rts, hops, S = _case(mode, S, D)
        for h, k in ((0, 10), (1, 4)):
            prev = hops[h - 1] if h else None
            win = S if h == 0 else 1
            got = block(hops[h], prev, roots, rts, win, k)
            want = M.block_loop(hops[h], prev, roots, rts, win, k)
            for f in ("indptr", "edge_dst", "edge_eid", "edge_dt", "src_nid", "src_ts"):
                if got[f].dtype != want[f].dtype or got[f].tobytes() != want[f].tobytes():
                    return False
            G, E = got["G"], got["E"]
            if E != int((hops[h].nbr >= 0).sum()) or len(got["src_nid"]) != G + E:
                return False
            src_t = got["src_ts"][G:].astype(np.float64)
            dst_t = got["src_ts"][got["edge_dst"]].astype(np.float64)
            if not np.all(src_t < dst_t):
                return False
            if got["edge_dt"].tobytes() != (got["src_ts"][got["edge_dst"]] - got["src_ts"][G:]).astype(np.float32).tobytes():
                return False
            if mode == "recent":
                for gidx in range(0, G, max(1, G // 50)):
                    a, b = got["indptr"][gidx], got["indptr"][gidx + 1]
                    if np.any(np.diff(src_t[a:b]) > 0):
                        return False
            if h == 1:
                valid1 = hops[0].nbr >= 0
                if got["src_nid"][:G].tobytes() != hops[0].nbr[valid1].tobytes():
                    return False
    return True


def test_block_pins():
    assert _checks(M.block)


def _inclusive(hop, prev, roots, rts, win, k):
    b = M.block(hop, prev, roots, rts, win, k)
    b["indptr"] = np.concatenate([b["indptr"][1:], b["indptr"][-1:]])
    return b


def _no_dst_prefix(hop, prev, roots, rts, win, k):
    b = M.block(hop, prev, roots, rts, win, k)
    b["src_nid"] = b["src_nid"][b["G"]:]
    b["src_ts"] = b["src_ts"][b["G"]:]
    return b


def _slot_dst(hop, prev, roots, rts, win, k):
    b = M.block(hop, prev, roots, rts, win, k)
    idx = np.flatnonzero(np.asarray(hop.nbr[:b["G"] * k]) >= 0)
    b["edge_dst"] = idx.astype(np.int64)
    return b


def _no_window_repeat(hop, prev, roots, rts, win, k):
    b = M.block(hop, prev, roots, rts, win, k)
    if prev is None and win > 1:
        G = b["G"]
        b["src_nid"] = np.concatenate([np.tile(np.asarray(roots, np.int32), win), b["src_nid"][G:]])
    return b


@pytest.mark.parametrize("mutant", [_inclusive, _no_dst_prefix, _slot_dst, _no_window_repeat])
def test_block_pins_catch_mutants(mutant):
    assert not _checks(mutant)
