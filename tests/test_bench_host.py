"""Host-side logic of the benchmark: the committed counter summaries it reads,
the spread of its timed steps over the epoch, and the all-core oracle timing
(root ranges per thread must find exactly the neighbours of one call)."""
import bench
from paper_2203_14883_amd import workloads as W


def test_profiles_match_the_current_kernels():
    """The committed summaries carry the hash of the kernel sources they were
    taken on; the benchmark uses them only while that hash is current."""
    h = bench.kernel_source_hash()
    for wl in ("c3", "c4", "c5"):
        prof = bench.read_profile(h, wl)
        assert prof is not None, wl
        assert prof["bytes"] > 0 and prof["avg_duration_us_under_counters"] > 0 and prof["slots_per_launch"] > 0
        f = bench.traffic_fields(prof)
        assert f["traffic"] == prof["bytes"]
        assert 0 < f["traffic_frac_in_counter_run"] < 1
    assert bench.read_profile("0" * 16, "c4") is None
    assert bench.traffic_fields(None) == {"traffic": None}


def test_step_positions_spread_over_the_epoch():
    for nb, B, n in [(325_000, 64, 20), (1_667, 1, 20), (263, 263, 20), (100, 64, 5), (10, 1, 1)]:
        pos = bench.step_positions(nb, B, n)
        assert len(pos) == n
        assert all(0 <= p <= max(nb - B, 0) for p in pos)
        assert pos == sorted(pos)
        if n > 1 and nb - B >= n:
            assert pos[0] == 0 and pos[-1] == nb - B and len(set(pos)) == n


def test_cpu_baseline_threads_agree_with_one_call():
    """A small Wikipedia-shaped workload: the oracle timed on one call and on
    root ranges over three threads (the function itself raises if the
    neighbour counts differ)."""
    w = W.make_c2(n_users=800, n_items=100, num_edges=8_000, seed=3)
    out = bench.cpu_baseline(w, 6, 3)
    assert out["cores"] == 3 and out["kind"] == "oracle" and out["unit"] == "neighbours/s"
    assert out["value"] > 0 and out["single_core"]["value"] > 0 and out["single_core"]["cores"] == 1
