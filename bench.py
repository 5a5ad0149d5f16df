#!/usr/bin/env python3
"""Benchmark of the temporal neighbour sampler on one MI355X.

Workload (default ``c4``): a MAG-shaped citation graph of 121.7M nodes and
1.3B edges (timestamps = publication years), undirected T-CSR of 2.6B
entries, 2-hop uniform sampling with fanouts 10x10, batches of 4,000 edges x 3
roots.  A step is one call of the sampler (all hops: window search, selection,
gather, compaction) over a super-batch of consecutive batches; the T-CSR is
built once before timing, as the paper builds it once per graph, and its build
time is reported beside the step rate.

Printed: one JSON line with sampled neighbours/s (valid slots of every hop per
second of sampler time), the roofline of the dominant kernel (the hop >= 2
sampling kernel, HIP events on its own stream), and the CPU oracle timed on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "sampled neighbours/sec (2-hop 10x10 uniform) + achieved HBM GB/s vs peak"


def log(msg):
    print("[bench %7.1fs] %s" % (time.time() - T0, msg), file=sys.stderr, flush=True)


T0 = time.time()


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=160,
                    help="timed steps (default 160: on c4, 160 x 64 batches spread over the epoch = 3.2%% of it)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c4", choices=["c2", "c3", "c4", "c5"])
    ap.add_argument("--batches-per-step", type=int, default=None,
                    help="batches fused into one sampler call (default: 64 for c3/c4, 1 for c5, 263 for c2)")
    ap.add_argument("--cpu-batches", type=int, default=None,
                    help="batches in the CPU oracle sample (default: eight steps' worth, about 10 s of oracle time on c4)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 4 GiB device copy (for scaling byte counters)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--small", action="store_true", help="reduced graph size (development only)")
    ap.add_argument("--row", default="sample", choices=["sample", "f1", "f2", "f4"],
                    help="sample: the sampler step (default); f1: node-feature lookup of the sampled slots; "
                         "f2: time encoding of the sampled slots; f4: MFG block export of the sampled hops")
    ap.add_argument("--gather-steps", type=int, default=8,
                    help="f1, f2: sampler steps whose slots are processed in the timed region")
    ap.add_argument("--consecutive", action="store_true",
                    help="time consecutive super-batches from the middle of the epoch (warm-up: the ones before)")
    ap.add_argument("--pointers", action="store_true",
                    help="hop 1 from saved window edges (Sec. 3.1 pointers), reset before warm-up; implies --consecutive")
    ap.add_argument("--chunk", type=int, default=None,
                    help="f1, f2: slots per launch (default 2^20 for f1, 2^23 for f2)")
    ap.add_argument("--epoch", action="store_true",
                    help="time every super-batch of the epoch in order (a full-epoch sweep; --steps is ignored)")
    ap.add_argument("--cpu-threads", type=int, default=None,
                    help="threads of the all-core oracle timing (default: the CPUs this process may use, "
                         "at most OMP_NUM_THREADS)")
    ap.add_argument("--no-dir", action="store_true",
                    help="build the T-CSR without its time directories (window searches use the index alone)")
    return ap.parse_args()


def strip_comments(src):
    """C++ source without comments, trailing blanks and empty lines (string
    and character literals are kept as they are)."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return "\n".join(l.rstrip() for l in "".join(out).splitlines() if l.strip())


def kernel_source_hash(files=("tgl_internal.hpp", "tgl_cells.hpp", "tgl_sample.hip")):
    """Hash of the code (comments left out) of the sources that define the
    measured kernels, to tell whether committed counters still apply."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2203_14883_amd", "csrc")
    for f in files:
        with open(os.path.join(csrc, f)) as fh:
            h.update(f.encode() + strip_comments(fh.read()).encode())
    return h.hexdigest()[:16]


def read_profile(kernel_hash, workload, prefix="hop_kernel"):
    """Figures of the committed counter summary of the dominant kernel
    (``profiles/<prefix>_<workload>_pmc.md``), if it was taken on the current
    kernel source: HBM bytes per launch and the launch duration measured in
    those same counter runs.  None otherwise."""
    name = "%s_%s_pmc.md" % (prefix, workload)
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if line.startswith("- ") and ":" in line:
            k, _, v = line[2:].partition(":")
            vals[k.strip()] = v.strip().strip("`")
    if vals.get("kernel_source_hash") != kernel_hash:
        return None
    try:
        out = {"bytes": float(vals["hbm_bytes_per_launch"]), "source": "profiles/" + name}
    except (KeyError, ValueError):
        return None
    for key, conv in (("avg_duration_us_under_counters", float), ("slots_per_launch", float)):
        try:
            out[key] = conv(vals[key])
        except (KeyError, ValueError):
            pass
    return out


def read_traffic(kernel_hash, workload, prefix="hop_kernel"):
    """HBM bytes per launch of a kernel from its committed counter summary
    (None unless taken on the current kernel source)."""
    prof = read_profile(kernel_hash, workload, prefix)
    return prof["bytes"] if prof else None


def traffic_fields(prof):
    """The byte counters' view of the dominant kernel, all from the counter
    runs themselves (bytes and duration of the same dispatches), never mixed
    with this run's timing."""
    if not prof:
        return {"traffic": None}
    f = {"traffic": prof["bytes"], "traffic_source": prof["source"]}
    us = prof.get("avg_duration_us_under_counters")
    if us:
        f["traffic_gbs_in_counter_run"] = prof["bytes"] / (us * 1e-6) / 1e9
        f["traffic_frac_in_counter_run"] = f["traffic_gbs_in_counter_run"] / PEAK_HBM_GBS
    if prof.get("slots_per_launch"):
        f["traffic_bytes_per_slot"] = prof["bytes"] / prof["slots_per_launch"]
    return f


def make_workload(name, small):
    from paper_2203_14883_amd import workloads as W
    if not small:
        return W.make(name)
    return {"c2": lambda: W.make_c2(),
            "c3": lambda: W.make_c3(num_edges=20_000_000),
            "c4": lambda: W.make_c4(num_nodes=12_170_000, num_edges=130_000_000),
            "c5": lambda: W.make_c5(num_nodes=1_000_000, num_edges=10_000_000)}[name]()


def step_positions(nb, B, n):
    """n super-batch start positions spread evenly over the epoch."""
    last = max(nb - B, 0)
    if n <= 1:
        return [last // 2]
    return [int(round(i * last / (n - 1))) for i in range(n)]


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.partition(":")[2].strip()
    except OSError:
        pass
    return "unknown CPU"


def cpu_threads(requested=None):
    """Threads for the all-core oracle timing: the CPUs this process may run
    on, at most OMP_NUM_THREADS when that is set."""
    if requested:
        return requested
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    cap = os.environ.get("OMP_NUM_THREADS")
    if cap and cap.isdigit() and int(cap) > 0:
        n = min(n, int(cap))
    return max(1, n)


def cpu_baseline(w, nbatches, threads):
    """The oracle as it stands (single-threaded C), on a bounded sample: the
    roots of ``nbatches`` consecutive batches from the middle of the epoch,
    over an oracle T-CSR that holds the full runs of every node the sample
    reaches.  Timed twice on the same roots: one call on one core, then the
    sample split into ``threads`` contiguous root ranges, one host thread
    each calling the unchanged oracle on its range with its own root_base
    (the sampler's output does not depend on how roots are batched; the
    ctypes call releases the interpreter lock).  Only sampling calls are
    timed."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    from oracle import subgraph
    nbatches = min(nbatches, w.num_batches())
    b0 = min(w.num_batches() // 2, w.num_batches() - nbatches)
    roots, rts, base = w.batches(b0, b0 + nbatches)
    src, dst, ts, eid = w.build_input()
    t = time.perf_counter()
    g = subgraph.reach_tcsr(src, dst, ts, eid, w.num_nodes, w.undirected, roots, rts, w.fanouts,
                            w.mode, w.snapshots, w.snapshot_len, w.sample_seed, base)
    build_s = time.perf_counter() - t
    log("CPU oracle: sub-graph of %d entries built in %.1f s" % (len(g.nbr), build_s))

    def valid(out):
        return int(sum(int((h.nbr >= 0).sum()) for h in out))

    t = time.perf_counter()
    out = oracle.sample(g, roots, rts, w.fanouts, w.mode, w.snapshots, w.snapshot_len,
                        w.sample_seed, base)
    dt1 = time.perf_counter() - t
    nbrs = valid(out)
    del out
    log("CPU oracle, 1 thread: %d neighbours in %.2f s" % (nbrs, dt1))

    # one contiguous range of roots per thread
    nt = max(1, min(threads, len(roots)))
    edges = [round(i * len(roots) / nt) for i in range(nt + 1)]
    ranges = [(edges[i], edges[i + 1]) for i in range(nt)]

    def work(rg):
        r0, r1 = rg
        return valid(oracle.sample(g, roots[r0:r1], rts[r0:r1], w.fanouts, w.mode, w.snapshots,
                                   w.snapshot_len, w.sample_seed, base + r0))

    t = time.perf_counter()
    with ThreadPoolExecutor(nt) as ex:
        counts = list(ex.map(work, ranges))
    dtn = time.perf_counter() - t
    if sum(counts) != nbrs:
        raise SystemExit("CPU oracle: %d threads found %d neighbours, one thread %d" % (nt, sum(counts), nbrs))
    log("CPU oracle, %d threads: %.2f s" % (nt, dtn))
    model = cpu_model()
    what = ("%d roots (%d consecutive batches from batch %d) of %s, %d hops, %d neighbours; T-CSR of the reached "
            "sub-graph (%d entries) built beforehand in %.1f s; sampling calls only; %s, %d logical CPUs on the host"
            % (len(roots), nbatches, b0, w.name, len(w.fanouts), nbrs, len(g.nbr), build_s, model,
               os.cpu_count() or 0))
    return dict(value=nbrs / dtn, unit="neighbours/s", cores=nt, kind="oracle",
                sample="%s; %d threads, each the unchanged single-threaded oracle on its own range of roots: %.2f s"
                       % (what, nt, dtn),
                cpu_model=model, host_logical_cpus=os.cpu_count(),
                single_core=dict(value=nbrs / dt1, unit="neighbours/s", cores=1, seconds=dt1))


GATHER_DIM = 768             # MAG node features (Table 3), bfloat16
GATHER_CHUNK = 1 << 22       # slots per tgl_gather launch (6.4 GB of rows)
GATHER_METRIC = "looked-up node-feature rows/sec (768-dim bf16) for the sampled slots + achieved HBM GB/s vs peak"


def gather_cpu_baseline(table, keys, nslots):
    """The lookup oracle, single-threaded, on a bounded sample: ``nslots``
    slots drawn at random from one step, over a host copy of exactly the table
    rows they reference (a full host copy of the table would not fit).  Only
    the oracle's lookup is timed."""
    import torch
    from oracle import features as F
    pick = np.sort(np.random.default_rng(2).choice(keys.numel(), min(nslots, keys.numel()), replace=False))
    k = keys[torch.from_numpy(pick).to(keys.device)].cpu().numpy().astype(np.int64)
    valid = (k >= 0) & (k < table.shape[0])
    uniq, inv = np.unique(k[valid], return_inverse=True)
    rows = table[torch.from_numpy(uniq).to(table.device)].view(torch.int16).cpu().numpy().view(np.uint16)
    kc = np.full(len(k), -1, np.int64)
    kc[valid] = inv
    t = time.perf_counter()
    (out,) = F.gather(kc.astype(np.int32), None, [(rows, F.NODE)])
    dt = time.perf_counter() - t
    return dict(value=len(k) / dt, unit="rows/s", cores=1, kind="oracle",
                sample="%d random slots of one c4 step (%d distinct nodes, %d PAD), %d-dim bf16 rows, %.2f s "
                       "single-threaded (lookup only; host copy of the referenced rows made beforehand)"
                       % (len(k), len(uniq), int((~valid).sum()), table.shape[1], dt))


def measure_gather(args, w, g, smp, run, timed_pos, B, dev):
    """Row f1: node-feature lookup (Fig. 2, steps 2-3) of every hop-1 and hop-2
    slot of sampler steps, GATHER_CHUNK slots per tgl_gather launch, against
    a table of GATHER_DIM-dim bf16 rows for every node of the graph."""
    import torch
    import paper_2203_14883_amd as P
    from oracle import features as F

    rows = w.num_nodes
    need = rows * GATHER_DIM * 2
    free, _ = torch.cuda.mem_get_info(dev)
    if need + (8 << 30) > free:
        raise SystemExit("f1: a %.1f GB feature table does not fit (%.1f GB free)" % (need / 1e9, free / 1e9))
    table = torch.empty((rows, GATHER_DIM), dtype=torch.bfloat16, device=dev)
    iv = table.view(torch.int16)
    gen = torch.Generator(device=dev)
    gen.manual_seed(12345)
    for i in range(0, rows, 1 << 22):
        iv[i:i + (1 << 22)].random_(-32768, 32767, generator=gen)   # random bits; values do not matter
    chunk = args.chunk or GATHER_CHUNK
    out = torch.empty((chunk, GATHER_DIM), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    log("f1: node-feature table %d x %d bf16 (%.1f GB)" % (rows, GATHER_DIM, need / 1e9))

    steps = timed_pos[:max(args.gather_steps, 1)]
    slot_lists = []                     # per step: the slots' neighbour ids of every hop, concatenated
    for b in steps:
        run(b)
        hs = smp.hops()
        slot_lists.append(torch.cat([h.nbr for h in hs]))
    torch.cuda.synchronize()

    def gather_all(keys):
        for c0 in range(0, keys.numel(), chunk):
            kc = keys[c0:c0 + chunk]
            P.gather(kc, None, [(table, "node")], outs=[out[:kc.numel()]])

    gather_all(slot_lists[0])           # warm-up
    torch.cuda.synchronize()
    P.timer_reset()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for keys in slot_lists:
        gather_all(keys)
    stop.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    k_ms, k_n = P.timer_read(P.binding.TIMER_GATHER)
    nslots = sum(int(k.numel()) for k in slot_lists)
    nvalid = sum(int(((k >= 0) & (k < rows)).sum()) for k in slot_lists)
    rb = GATHER_DIM * 2
    alg_bytes = nslots * (4 + rb) + nvalid * rb        # key read + row written per slot; row read when valid
    achieved = alg_bytes / k_n / (k_ms / k_n * 1e-3) / 1e9
    value = nslots / (total_ms * 1e-3)
    log("f1: %d launches, %d slots (%d valid): %.2f ms total, kernel %.2f ms; %.3g rows/s; %.1f GB/s algorithmic"
        % (k_n, nslots, nvalid, total_ms, k_ms, value, achieved))

    # parity spot check of the last launch against the oracle (sampled rows)
    last = slot_lists[-1]
    c0 = ((last.numel() - 1) // chunk) * chunk
    kc = last[c0:]
    pick = torch.from_numpy(np.random.default_rng(1).choice(kc.numel(), min(4096, kc.numel()), replace=False)).to(dev)
    keys = kc[pick].cpu().numpy()
    ok = (keys >= 0) & (keys < rows)
    uniq, inv = np.unique(keys[ok], return_inverse=True)
    host_rows = table[torch.from_numpy(uniq.astype(np.int64)).to(dev)].view(torch.int16).cpu().numpy().view(np.uint16)
    kk = np.full(len(keys), -1, np.int32)
    kk[ok] = inv
    (want,) = F.gather(kk, None, [(host_rows, F.NODE)])
    got = out[pick].view(torch.int16).cpu().numpy().view(np.uint16)
    if got.tobytes() != want.tobytes():
        raise SystemExit("f1: looked-up rows differ from the oracle")
    log("f1: %d sampled rows of the last launch equal the oracle's" % len(keys))

    cpu = None
    if not args.no_cpu_baseline:
        del out
        torch.cuda.empty_cache()
        cpu = gather_cpu_baseline(table, slot_lists[len(slot_lists) // 2], 2 << 20)
        log("f1 CPU oracle: %.3g rows/s (%s)" % (cpu["value"], cpu["sample"]))
    khash = kernel_source_hash(("tgl_internal.hpp", "tgl_gather.hip"))
    line = {
        "metric": GATHER_METRIC,
        "value": value,
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": len(slot_lists),
        "warmup": 1,
        "ms_per_step": total_ms / len(slot_lists),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "%s: node-feature lookup (%d-dim bf16 rows, %d nodes) of every hop-1 and hop-2 slot of %d "
                        "sampler steps (%d-hop %s %s, %d batches of %d edges x 3 roots per step), %d slots per launch"
                        % (w.name, GATHER_DIM, rows, len(slot_lists), len(w.fanouts), w.mode,
                           "x".join(map(str, w.fanouts)), B, w.batch_edges, chunk),
            "slots_per_step": nslots / len(slot_lists),
            "valid_fraction": nvalid / max(nslots, 1),
        },
        "roofline": {
            "kernel": "gather_kernel",
            "bound": "hbm",
            "achieved": achieved,
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS,
            "traffic": read_traffic(khash, w.name, "gather_kernel"),
            "algorithmic_bytes_per_launch": alg_bytes / k_n,
            "avg_launch_ms": k_ms / k_n,
            "kernel_source_hash": khash,
        },
        "cpu_baseline": cpu,
    }
    P.timer_disable()
    print(json.dumps(line), flush=True)


TIME_DIM = 100               # time-encoding width (TGL's default)
TIME_CHUNK = 1 << 23          # slots per tgl_time_encode launch (3.2 GB of float32 rows)
TIME_METRIC = "time-encoded slots/sec (100-dim float32, Eq. 3) for the sampled slots + achieved HBM GB/s vs peak"


def measure_timeenc(args, w, smp, run, timed_pos, B, dev):
    """Row f2: time encoding (Eq. 3) of the dt of every hop-1 and hop-2 slot
    of sampler steps, TIME_CHUNK slots per tgl_time_encode launch, float32
    rows of TIME_DIM elements, TGAT-style frequencies omega_j = 10^(-9j/(d-1))."""
    import torch
    import paper_2203_14883_amd as P
    from oracle import features as F

    omega_h = (1.0 / 10 ** np.linspace(0, 9, TIME_DIM)).astype(np.float32)
    phi_h = (np.random.default_rng(7).random(TIME_DIM) * 6.0 - 3.0).astype(np.float32)
    omega, phi = torch.from_numpy(omega_h).to(dev), torch.from_numpy(phi_h).to(dev)
    chunk = args.chunk or TIME_CHUNK
    out = torch.empty((chunk, TIME_DIM), dtype=torch.float32, device=dev)
    steps = timed_pos[:max(args.gather_steps, 1)]
    dts = []
    for b in steps:
        run(b)
        dts.append(torch.cat([h.dt for h in smp.hops()]))
    torch.cuda.synchronize()

    def encode_all(d):
        for c0 in range(0, d.numel(), chunk):
            dc = d[c0:c0 + chunk]
            P.time_encode(dc, omega, phi, out=out[:dc.numel()])

    encode_all(dts[0])                  # warm-up
    torch.cuda.synchronize()
    P.timer_reset()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for d in dts:
        encode_all(d)
    stop.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    k_ms, k_n = P.timer_read(P.binding.TIMER_TIMEENC)
    nslots = sum(int(d.numel()) for d in dts)
    nvalid = sum(int((d >= 0).sum()) for d in dts)
    alg_bytes = nslots * (4 + TIME_DIM * 4)          # dt read, row written
    achieved = alg_bytes / k_n / (k_ms / k_n * 1e-3) / 1e9
    value = nslots / (total_ms * 1e-3)
    log("f2: %d launches, %d slots (%d valid): %.2f ms total, kernel %.2f ms; %.3g slots/s; %.1f GB/s algorithmic"
        % (k_n, nslots, nvalid, total_ms, k_ms, value, achieved))

    # spot check of the last launch against the oracle (sampled rows, derived tolerance)
    last = dts[-1]
    c0 = ((last.numel() - 1) // chunk) * chunk
    dc = last[c0:]
    pick = np.random.default_rng(1).choice(dc.numel(), min(4096, dc.numel()), replace=False)
    pk = torch.from_numpy(pick).to(dev)
    want = F.time_encode(dc[pk].cpu().numpy(), omega_h, phi_h)
    got = out[pk].cpu().numpy().astype(np.float64)
    err = float(np.abs(got - want).max()) if want.size else 0.0
    if not err <= 1e-6:
        raise SystemExit("f2: encodings differ from the oracle by %.3g" % err)
    log("f2: %d sampled rows of the last launch within %.2g of the oracle" % (len(pick), err))

    cpu = None
    if not args.no_cpu_baseline:
        d = dts[len(dts) // 2]
        pick = np.sort(np.random.default_rng(2).choice(d.numel(), min(1 << 20, d.numel()), replace=False))
        dh = d[torch.from_numpy(pick).to(dev)].cpu().numpy()
        t = time.perf_counter()
        F.time_encode(dh, omega_h, phi_h)
        dt_ = time.perf_counter() - t
        cpu = dict(value=len(dh) / dt_, unit="slots/s", cores=1, kind="oracle",
                   sample="%d random slots of one c4 step, %d-dim rows, %.2f s single-threaded (numpy float64)"
                          % (len(dh), TIME_DIM, dt_))
        log("f2 CPU oracle: %.3g slots/s (%s)" % (cpu["value"], cpu["sample"]))
    khash = kernel_source_hash(("tgl_internal.hpp", "tgl_timeenc.hip"))
    line = {
        "metric": TIME_METRIC,
        "value": value,
        "unit": "slots/s",
        "n_gpus": 1,
        "steps": len(dts),
        "warmup": 1,
        "ms_per_step": total_ms / len(dts),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "%s: time encoding (%d-dim float32 rows) of every hop-1 and hop-2 slot of %d sampler steps "
                        "(%d-hop %s %s, %d batches of %d edges x 3 roots per step), %d slots per launch"
                        % (w.name, TIME_DIM, len(dts), len(w.fanouts), w.mode, "x".join(map(str, w.fanouts)),
                           B, w.batch_edges, chunk),
            "slots_per_step": nslots / len(dts),
            "valid_fraction": nvalid / max(nslots, 1),
        },
        "roofline": {
            "kernel": "timeenc_vec_kernel",
            "bound": "hbm",
            "achieved": achieved,
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS,
            "traffic": read_traffic(khash, w.name, "timeenc_kernel"),
            "algorithmic_bytes_per_launch": alg_bytes / k_n,
            "avg_launch_ms": k_ms / k_n,
            "kernel_source_hash": khash,
        },
        "cpu_baseline": cpu,
    }
    P.timer_disable()
    print(json.dumps(line), flush=True)


MFG_METRIC = "exported MFG edges/sec (CSC blocks of every hop of the sampler step) + achieved HBM GB/s vs peak"


def measure_mfg(args, w, smp, run, inputs, timed_pos, B, dev):
    """Row f4: the MFG blocks (Alg. 1, "generate DGL MFGs") of every hop of
    sampler steps, exported on the device; only the export kernels are timed
    (HIP events around each export).  Algorithmic bytes per hop: per slot its
    nbr read; per group its valid count written and read, its indptr entry
    and destination node written (and, after hop 1, its parent and the
    parent slot's node and time read); per edge the slot's eid, ts, dt read
    and the edge's dst, eid, dt and source node and time written."""
    import torch
    import paper_2203_14883_amd as P
    from oracle import mfg as M

    steps = timed_pos[:max(args.gather_steps, 1)]
    run(steps[0])
    r, t_, _, _ = inputs[steps[0]]
    for h in range(len(w.fanouts)):
        P.mfg_export(smp, h, r, t_)                  # warm-up
    torch.cuda.synchronize()
    P.timer_reset()
    alg = 0.0
    nedges = 0
    launches = 0
    blocks = None
    for b in steps:
        run(b)
        r, t_, _, _ = inputs[b]
        blocks = [P.mfg_export(smp, h, r, t_) for h in range(len(w.fanouts))]
        hs = smp.hops()                              # syncs: sizes for the byte count
        for h, (hop, blk) in enumerate(zip(hs, blocks)):
            G, E = (int(v) for v in blk.sizes.cpu().tolist())
            slots = hop.nbr.numel()
            alg += slots * 4 + G * (4 + 4 + 8 + 8) + (G * (8 + 8) if h else 0) + E * (16 + 8 + 8 + 4 + 4 + 4)
            nedges += E
            launches += 1
    k_ms, k_n = P.timer_read(P.binding.TIMER_MFG)
    achieved = alg / (k_ms * 1e-3) / 1e9
    value = nedges / (k_ms * 1e-3)
    log("f4: %d exports, %d edges: kernels %.2f ms; %.3g edges/s; %.1f GB/s algorithmic"
        % (k_n, nedges, k_ms, value, achieved))

    # properties of the last step's blocks that hold at any size
    hs = smp.hops()
    for h, (hop, blk) in enumerate(zip(hs, blocks)):
        s = blk.sliced()
        G, E = (int(v) for v in s.sizes.cpu().tolist())
        valid = hop.nbr >= 0
        ok = E == int(valid.sum()) and int(s.indptr[-1]) == E and bool((s.indptr[1:] >= s.indptr[:-1]).all())
        pick = torch.from_numpy(np.random.default_rng(h).choice(E, min(E, 4096), replace=False)).to(dev) if E else None
        if ok and E:
            src_t = s.src_ts[G + pick].double()
            dst_t = s.src_ts[s.edge_dst[pick]].double()
            ok = bool((src_t < dst_t).all())
            slot_idx = torch.nonzero(valid).flatten()[pick]
            ok = ok and torch.equal(s.edge_eid[pick], hop.eid[slot_idx]) and torch.equal(s.src_nid[G + pick], hop.nbr[slot_idx])
        if not ok:
            raise SystemExit("f4: block of hop %d fails its invariants" % (h + 1))
    log("f4: blocks of the last step satisfy the size, order and slot invariants")

    cpu = None
    if not args.no_cpu_baseline:
        # oracle block of hop 2 of a bounded sample: the first 2^20 hop-2 groups' slots of the last step,
        # given as host arrays (their values are not checked here, only the oracle's time is taken)
        hop = hs[-1]
        k = w.fanouts[-1]
        ng = min(hop.num_roots, 1 << 20)

        class _H:
            pass
        hh = _H()
        hh.nbr, hh.eid = hop.nbr[:ng * k].cpu().numpy(), hop.eid[:ng * k].cpu().numpy()
        hh.ts, hh.dt = hop.ts[:ng * k].cpu().numpy(), hop.dt[:ng * k].cpu().numpy()
        hh.parent, hh.num_roots = hop.parent[:ng].cpu().numpy(), ng
        pp = _H()
        pp.nbr, pp.ts = hs[-2].nbr.cpu().numpy(), hs[-2].ts.cpu().numpy()
        t = time.perf_counter()
        out = M.block(hh, pp, None, None, 1, k)
        dt_ = time.perf_counter() - t
        cpu = dict(value=out["E"] / dt_, unit="edges/s", cores=1, kind="oracle",
                   sample="hop-2 block of the first %d groups of one c4 step (%d edges), %.2f s single-threaded (numpy)"
                          % (ng, out["E"], dt_))
        log("f4 CPU oracle: %.3g edges/s (%s)" % (cpu["value"], cpu["sample"]))
    khash = kernel_source_hash(("tgl_internal.hpp", "tgl_mfg.hip"))
    line = {
        "metric": MFG_METRIC,
        "value": value,
        "unit": "edges/s",
        "n_gpus": 1,
        "steps": len(steps),
        "warmup": 1,
        "ms_per_step": k_ms / len(steps),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {
            "workload": "%s: MFG blocks (CSC) of every hop of %d sampler steps (%d-hop %s %s, %d batches of %d edges "
                        "x 3 roots per step)" % (w.name, len(steps), len(w.fanouts), w.mode,
                                                 "x".join(map(str, w.fanouts)), B, w.batch_edges),
            "edges_per_step": nedges / len(steps),
        },
        "roofline": {
            "kernel": "tgl_mfg_export (count, scan, scatter)",
            "bound": "hbm",
            "achieved": achieved,
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS,
            "traffic": read_traffic(khash, w.name, "mfg_export"),
            "algorithmic_bytes_per_launch": alg / max(launches, 1),
            "avg_launch_ms": k_ms / max(k_n, 1),
            "kernel_source_hash": khash,
        },
        "cpu_baseline": cpu,
    }
    P.timer_disable()
    print(json.dumps(line), flush=True)


def copy_calibration(dev, gib=4, reps=3):
    """A plain device copy of known size, so byte counters can be scaled."""
    import torch
    n = gib << 30
    a = torch.empty(n, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    a.fill_(1)
    torch.cuda.synchronize()
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    del a, b
    torch.cuda.empty_cache()
    return dict(bytes_read=n, bytes_written=n, reps=reps)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only (this build has no multi-GPU path); got --gpus %d"
              % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2203_14883_amd as P

    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        sys.exit(1)
    P.lib()   # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.copy_calibration:
        log("copy calibration: %s" % copy_calibration(dev))
    log("generating workload %s%s" % (args.workload, " (small)" if args.small else ""))
    w = make_workload(args.workload, args.small)
    log("graph: %d nodes, %d edges" % (w.num_nodes, w.num_edges))

    src, dst, ts, eid = w.build_input()
    d_src = torch.from_numpy(src).to(dev)
    d_dst = torch.from_numpy(dst).to(dev)
    d_ts = torch.from_numpy(ts).to(dev)
    d_eid = None if eid is None else torch.from_numpy(eid).to(dev)
    torch.cuda.synchronize()
    log("COO uploaded")

    ws = torch.empty(P.tcsr_build_workspace(w.num_edges, w.num_nodes, w.undirected),
                     dtype=torch.uint8, device=dev)
    # neighbour histories serve the hops >= 2 of a sampler with one window
    # unbounded below; other samplers never read them, and the rows after the
    # sampler (f1, f2, f4) only need its slots (f1's feature table needs the
    # memory)
    hist = (args.row == "sample" and len(w.fanouts) > 1 and w.snapshots == 1
            and math.isinf(w.snapshot_len))
    # time directories serve the window searches of long runs; with
    # histories only hop 1 searches, which for c4's runs (mostly short, a
    # single edge per root) measured the same with and without them
    tdir = args.row == "sample" and not hist and not args.no_dir
    P.timer_enable(1 << 14)
    g = P.tcsr_build(d_src, d_dst, d_ts, d_eid, w.num_nodes, w.undirected, workspace=ws, hist=hist,
                     dir=tdir)  # warm-up
    del g
    torch.cuda.synchronize()
    P.timer_reset()
    t = time.perf_counter()
    g = P.tcsr_build(d_src, d_dst, d_ts, d_eid, w.num_nodes, w.undirected, workspace=ws, hist=hist, dir=tdir)
    torch.cuda.synchronize()
    build_wall = time.perf_counter() - t
    build_ms, _ = P.timer_read(P.binding.TIMER_BUILD)
    del ws, d_src, d_dst, d_ts, d_eid
    torch.cuda.empty_cache()
    log("T-CSR built: %d entries%s, %.1f ms (events), %.1f ms wall"
        % (g.num_entries, " with neighbour histories" if hist else "", build_ms, build_wall * 1e3))

    B = args.batches_per_step or {"c2": w.num_batches(), "c3": 64, "c4": 64, "c5": 1}[args.workload]
    B = min(B, w.num_batches())
    if args.epoch:
        # every super-batch of the epoch, in order; warm-up on the first ones
        timed_pos = list(range(0, w.num_batches(), B))
        warm_pos = timed_pos[:args.warmup]
        args.steps = len(timed_pos)
    elif args.consecutive or args.pointers:
        # consecutive super-batches in chronological order, warm-up steps right before them
        nsteps = args.warmup + args.steps
        b0 = max(0, min(w.num_batches() // 2 - (nsteps * B) // 2, w.num_batches() - nsteps * B))
        if b0 + nsteps * B > w.num_batches():
            raise SystemExit("--consecutive: the epoch has fewer than %d super-batches of %d batches" % (nsteps, B))
        warm_pos = [b0 + i * B for i in range(args.warmup)]
        timed_pos = [b0 + (args.warmup + i) * B for i in range(args.steps)]
    else:
        # timed steps are spread evenly over the epoch; warm-up steps sit between them
        timed_pos = step_positions(w.num_batches(), B, args.steps)
        span = max(w.num_batches() - B, 1)
        warm_pos = [(p + max(span // (2 * max(args.steps, 1)), 1)) % span for p in timed_pos[:args.warmup]]
    inputs = {}
    for b in sorted(set(timed_pos + warm_pos)):
        r, t_, base = w.batches(b, min(b + B, w.num_batches()))
        inputs[b] = (torch.from_numpy(r).to(dev), torch.from_numpy(t_).to(dev), base, len(r))
    max_roots = max(v[3] for v in inputs.values())
    smp = P.Sampler(max_roots, w.fanouts, w.snapshots, device=dev)
    log("sampler buffers: %d roots per step, %.2f GB outputs+workspace"
        % (max_roots, sum(x.numel() * x.element_size() for x in
                          smp.nbr + smp.eid + smp.ts + smp.dt + [smp.workspace]) / 1e9))

    ptr = P.pointers_reset(g, w.snapshots) if args.pointers else None

    def run(b):
        r, t_, base, n = inputs[b]
        smp.run(g, r, t_, w.mode, w.snapshot_len, w.sample_seed, base, num_roots=n, pointers=ptr)

    if args.row == "f1":
        measure_gather(args, w, g, smp, run, timed_pos, B, dev)
        return
    if args.row == "f2":
        measure_timeenc(args, w, smp, run, timed_pos, B, dev)
        return
    if args.row == "f4":
        measure_mfg(args, w, smp, run, inputs, timed_pos, B, dev)
        return

    for b in warm_pos:
        run(b)
    torch.cuda.synchronize()
    # Inside the timed region only the dominant kernel (hops >= 2; hop 1 for
    # one-hop samplers) carries timer events: every event pair between kernels
    # costs the step time (3% on c4 with all of them).
    dominant = P.binding.TIMER_HOPN if len(w.fanouts) > 1 else P.binding.TIMER_HOP1
    P.timer_reset()
    P.timer_select(dominant)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for b in timed_pos:
        run(b)
    stop.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    dom_ms, dom_n = P.timer_read(dominant)
    P.timer_select()
    P.timer_reset()

    # untimed pass over the same steps: valid slots (neighbours), the
    # algorithmic bytes of the dominant kernel (every hop >= 2; hop 1 of a
    # one-hop sampler), and the other kernels' times
    indptr = g.indptr
    nbrs_total = 0
    slots_total = 0
    dom_bytes = 0.0
    dom_slots = 0
    dom_roots = 0
    bounds_h1 = 1 if math.isinf(w.snapshot_len) else w.snapshots + 1
    bounds_hn = 1 if math.isinf(w.snapshot_len) else 2

    def search_bytes(x, nb):
        """4 bytes per probe of a binary search over each root's run, nb
        window edges per root (nodes outside the graph search nothing)."""
        ok = (x >= 0) & (x < w.num_nodes)
        xs = x[ok]
        deg = (indptr[xs + 1] - indptr[xs]).double()
        return float((torch.ceil(torch.log2(deg + 1.0)) * 4.0 * nb).sum())

    for b in timed_pos:
        run(b)
        hs = smp.hops()
        for h, hop in enumerate(hs):
            valid = hop.nbr >= 0
            nv = int(valid.sum())
            nbrs_total += nv
            slots_total += hop.nbr.numel()
            if h >= 1:
                dom_slots += hop.nbr.numel()
                dom_roots += hop.num_roots
                roots2 = hs[h - 1].nbr[hs[h - 1].nbr >= 0].long()
                # per root: node + time read, run bounds read, parent index written;
                # per slot: 16-byte entry read when valid, 20 bytes written
                dom_bytes += (hop.num_roots * (8 + 16 + 8) + search_bytes(roots2, bounds_hn) + nv * 16
                              + hop.nbr.numel() * 20)
            elif dominant == P.binding.TIMER_HOP1:
                r, _, _, n = inputs[b]
                dom_slots += hop.nbr.numel()
                dom_roots += n
                # per root: node + time read, run bounds read; S + 1 window
                # edges searched (one when windows are unbounded below); per
                # slot as above
                dom_bytes += n * (8 + 16) + search_bytes(r[:n].long(), bounds_h1) + nv * 16 + hop.nbr.numel() * 20
    hop1_ms, hop1_n = P.timer_read(P.binding.TIMER_HOP1)
    comp_ms, comp_n = P.timer_read(P.binding.TIMER_COMPACT)
    if dominant == P.binding.TIMER_HOP1:
        hop1_ms, hop1_n = dom_ms, dom_n
    log("timed %d steps: %.2f ms total (timed region: %s %.2f ms; recount pass: hop1 %.2f, compaction %.2f ms)"
        % (args.steps, total_ms, "hopN" if dominant == P.binding.TIMER_HOPN else "hop1", dom_ms,
           hop1_ms, comp_ms))
    dom_bytes_per_launch = dom_bytes / max(dom_n, 1)
    dom_slots_per_launch = dom_slots / max(dom_n, 1)
    avg_dom_ms = dom_ms / max(dom_n, 1)
    achieved = dom_bytes_per_launch / (avg_dom_ms * 1e-3) / 1e9 if avg_dom_ms > 0 else 0.0
    value = nbrs_total / (total_ms * 1e-3)
    khash = kernel_source_hash()
    prof = read_profile(khash, args.workload) if not (args.small or args.epoch) else None
    if len(w.fanouts) > 1:
        kernel = "hop_single_kernel (hops >= 2)"
    elif w.snapshots > 1:
        kernel = "hop_multi_kernel (hop 1)" if w.snapshots <= 8 else "hop_multi_wide_kernel (hop 1)"
    else:
        kernel = "hop_single_kernel (hop 1)"
    log("neighbours %d over %d slots; %.3g neighbours/s; %s %.1f GB/s algorithmic"
        % (nbrs_total, slots_total, value, kernel, achieved))

    cpu = None
    if not args.no_cpu_baseline:
        log("CPU oracle baseline")
        cpu = cpu_baseline(w, args.cpu_batches or min(8 * B, 512), cpu_threads(args.cpu_threads))
        log("CPU oracle: %.3g neighbours/s on %d threads, %.3g on one (%s)"
            % (cpu["value"], cpu["cores"], cpu["single_core"]["value"], cpu["sample"]))
        if args.workload == "c5":
            # c5's T-CSR is built from a shuffled COO: the oracle's build of the
            # same COO, on one core, beside the GPU build
            import oracle
            src, dst, ts, eid = w.build_input()
            t = time.perf_counter()
            og = oracle.build_tcsr(src, dst, ts, eid, w.num_nodes, w.undirected)
            cpu["build"] = dict(seconds=time.perf_counter() - t, entries=len(og.nbr), cores=1,
                                gpu_ms=build_ms, what="oracle_build of the same shuffled COO")
            log("CPU oracle build of the %d-entry T-CSR from the shuffled COO: %.1f s (GPU: %.1f ms)"
                % (len(og.nbr), cpu["build"]["seconds"], build_ms))
            del og, src, dst, ts, eid

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "neighbours/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": total_ms / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "%s%s: %d nodes, %d edges, undirected T-CSR of %d entries; %d-hop %s %s, %d snapshot(s)%s; %d batches of %d edges x 3 roots per step%s"
                        % (w.name, " (reduced)" if args.small else "", w.num_nodes, w.num_edges,
                           g.num_entries, len(w.fanouts), w.mode, "x".join(map(str, w.fanouts)),
                           w.snapshots, "" if math.isinf(w.snapshot_len) else " of %g" % w.snapshot_len,
                           B, w.batch_edges,
                           "; full epoch (%d batches)" % w.num_batches() if args.epoch else ""),
            "roots_per_step": max_roots,
            "step_order": ("the whole epoch in order" if args.epoch else
                           "consecutive" if (args.consecutive or args.pointers) else "spread over the epoch"),
            "hop1_pointers": bool(args.pointers),
            "neighbours_per_step": nbrs_total / args.steps,
            "slots_per_step": slots_total / args.steps,
            "tcsr_build_ms": build_ms,
            "tcsr_neighbour_histories": bool(hist),
            "tcsr_time_directory": bool(tdir),
            "kernel_ms_per_step": {"hop1": hop1_ms / args.steps, "hopN": (dom_ms if dominant == P.binding.TIMER_HOPN
                                                                          else 0.0) / args.steps,
                                   "compaction": comp_ms / args.steps,
                                   "timed_in_region": "hopN" if dominant == P.binding.TIMER_HOPN else "hop1"},
        },
        "roofline": {
            "kernel": kernel,
            "bound": "hbm",
            "achieved": achieved,
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS,
            **traffic_fields(prof),
            "algorithmic_bytes_per_slot": dom_bytes_per_launch / dom_slots_per_launch if dom_slots_per_launch else None,
            "algorithmic_bytes_per_launch": dom_bytes_per_launch,
            "roots_per_launch": dom_roots / max(dom_n, 1),
            "slots_per_launch": dom_slots_per_launch,
            "avg_launch_ms": avg_dom_ms,
            "launches": dom_n,
            "kernel_source_hash": khash,
        },
        "cpu_baseline": cpu,
    }
    P.timer_disable()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
