"""Planted mistakes in the oracle (on the CPU): each mutant of tgl_oracle.c
must be caught by at least one pin.  This shows that the pins are sensitive
to the plausible slips -- a dropped term, a flipped comparison, a wrong index
or operand order -- and not only to crashes."""
import math
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
from oracle import brute
from checks import assert_hops_equal
from golden_io import floats, ints, read

SRC = os.path.join(os.path.dirname(oracle.__file__), "tgl_oracle.c")

MUTANTS = {
    "non_strict_time": ("if ((double)ts[mid] < v) lo = mid + 1;", "if ((double)ts[mid] <= v) lo = mid + 1;"),
    "tie_order_reversed": ("if (ent[j].t < ent[i].t) tmp[k++] = ent[j++];", "if (ent[j].t <= ent[i].t) tmp[k++] = ent[j++];"),
    "merge_skip_wrong": ("if (!(ent[mid].t < ent[mid - 1].t)) continue;", "if (!(ent[mid].t < ent[lo].t)) continue;"),
    "most_recent_oldest_first": ("if (j < n) p = hi - 1 - j;", "if (j < n) p = lo + j;"),
    "child_path_drops_window": ("+ (uint64_t)s * (uint64_t)k + (uint64_t)j", "+ (uint64_t)j"),
    "window_low_bound_off_by_one": ("(double)(s + 1) * (double)delta", "(double)(s + 2) * (double)delta"),
    "dt_sign": ("(float)((double)ct[q] - (double)ts[p])", "(float)((double)ts[p] - (double)ct[q])"),
    "hash_key_shift": ("(uint64_t)(uint32_t)hop << 40", "(uint64_t)(uint32_t)hop << 41"),
    "mix_constant": ("0xBF58476D1CE4E5B9ULL", "0xBF58476D1CE4E5B8ULL"),
    "reversed_neighbour": ("en.v = fwd ? dst[k] : src[k];", "en.v = dst[k];"),
    "negative_zero_kept": ("en.t = ts[k] == 0.0f ? 0.0f : ts[k];", "en.t = ts[k];"),
    "draw_by_modulo": ("if (n > 0) p = lo + scale_draw(oracle_slot_hash(seed, cp[q], h, s, j), n);",
                       "if (n > 0) p = lo + (int64_t)(oracle_slot_hash(seed, cp[q], h, s, j) % (uint64_t)n);"),
    "child_forgets_window": ("int32_t s = (h == 1) ? w : cs[q];", "int32_t s = (h == 1) ? w : 0;"),
    "indptr_shifted": ("indptr[u + 1] += 1;", "indptr[u] += 1;"),
    "hash_hop_index": ("oracle_slot_hash(seed, cp[q], h, s, j)", "oracle_slot_hash(seed, cp[q], h - 1, s, j)"),
    "parent_is_root": ("o_parent[h][n_next] = slot;", "o_parent[h][n_next] = q;"),
    "window_top_ignores_snapshot": ("return (double)t - (double)s * (double)delta;", "return (double)t;"),
}


def _pins(lib):
    """Run a fast subset of the pins against ``lib``; returns the names that failed."""
    failed = []
    # published SplitMix64 vector
    if lib.oracle_mix64(0x9E3779B97F4A7C15) != 0xE220A8397B1DCDAF:
        failed.append("mix64")
    # hand-worked golden example
    G = read("fig3_tcsr.txt")
    for kind in ("directed", "undirected"):
        g = oracle.build_tcsr(ints(G["coo_src"]), ints(G["coo_dst"]), floats(G["coo_ts"]),
                              ints(G["coo_eid"]), 5, kind == "undirected", lib=lib)
        if not (np.array_equal(g.nbr, ints(G[kind + ".nbr"])) and
                np.array_equal(g.indptr, ints(G[kind + ".indptr"]))):
            failed.append("golden-" + kind)
    # brute force on random tiny graphs
    rng = np.random.default_rng(99)
    for trial in range(60):
        N = int(rng.integers(1, 25))
        m0 = int(rng.integers(0, 150))
        src = rng.integers(0, N, m0).astype(np.int32)
        dst = rng.integers(0, N, m0).astype(np.int32)
        ts = rng.integers(0, 20, m0).astype(np.float32)
        if m0:
            ts[rng.integers(0, m0, max(1, m0 // 8))] = -0.0
        und = bool(trial % 2)
        R = int(rng.integers(1, 10))
        roots = rng.integers(0, N, R).astype(np.int32)
        rts = rng.integers(0, 24, R).astype(np.float32)
        fan = [int(rng.choice([1, 3, 10])) for _ in range(int(rng.integers(1, 4)))]
        mode = ["recent", "uniform"][trial % 4 // 2]
        S = int(rng.integers(1, 4))
        delta = float(rng.choice([2.0, 5.0])) if S > 1 or trial % 3 else math.inf
        try:
            g = oracle.build_tcsr(src, dst, ts, None, N, und, lib=lib)
            got = oracle.sample(g, roots, rts, fan, mode, S, delta, 5, 17, lib=lib)
            want = brute.sample(src, dst, ts, None, N, und, roots, rts, fan, mode, S, delta, 5, 17)
            assert_hops_equal(got, want)
        except Exception:
            failed.append("brute")
            break
    return failed


def test_unmutated_oracle_passes_pins():
    assert _pins(oracle.load()) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    """Each mutant runs in a child process: a mutant that corrupts memory and
    crashes is caught as surely as one that returns wrong values."""
    old, new = MUTANTS[name]
    text = open(SRC).read()
    assert text.count(old) == 1, "mutation anchor not found: " + name
    mpath = tmp_path / ("mut_%s.c" % name)
    mpath.write_text(text.replace(old, new))
    so = oracle.compile_oracle(str(mpath), str(tmp_path / ("mut_%s.so" % name)))
    here = os.path.dirname(os.path.abspath(__file__))
    code = ("import sys; sys.path[:0] = [%r, %r]\n"
            "import oracle, test_oracle_mutants as T\n"
            "sys.exit(1 if T._pins(oracle.load(%r)) else 0)\n") % (here, os.path.dirname(here), str(so))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, "mutant %s survived every pin" % name
