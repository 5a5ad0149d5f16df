"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/tgl.h declares, sizes its buffers consistently, and
rejects invalid arguments before touching the device."""
import ctypes as C
import math
import os
import re

import numpy as np
import pytest

import paper_2203_14883_amd as P
from paper_2203_14883_amd import binding as B

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "tgl.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tgl_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_function():
    names = declared_functions()
    assert set(names) == set(B.EXPORTS)
    L = P.lib()
    for n in names:
        assert hasattr(L, n), n
    assert L.tgl_version() == 10000


def test_status_strings():
    for s in (0, -1, -2, -3, -4):
        assert P.status_str(s) and P.status_str(s) != "unknown status"
    assert P.status_str(7) == "unknown status"


def _fan(v):
    a = np.asarray(v, np.int32)
    return a, a.ctypes.data_as(C.c_void_p)


def test_capacity_and_workspace():
    L = P.lib()
    a, p = _fan([10, 10])
    assert L.tgl_sample_capacity(12000, 2, p, 1, 0) == 12000
    assert L.tgl_sample_capacity(12000, 2, p, 1, 1) == 120000
    assert L.tgl_sample_capacity(12000, 2, p, 1, 2) == 1200000
    assert L.tgl_sample_capacity(180000, 2, p, 3, 2) == 180000 * 3 * 100
    assert L.tgl_sample_capacity(10, 2, p, 1, 3) == -1
    a, p = _fan([1024] * 8)
    assert L.tgl_sample_capacity(10**6, 8, p, 1, 8) == -1          # beyond 2^62
    assert L.tgl_sample_workspace(10**6, 8, p, 1) == 0
    a, p = _fan([10])
    assert L.tgl_sample_workspace(100, 1, p, 1) > 0                  # single hop: token size
    a, p = _fan([10, 10, 10])
    w2 = L.tgl_sample_workspace(1000, 2, _fan([10, 10])[1], 1)
    w3 = L.tgl_sample_workspace(1000, 3, p, 1)
    assert w3 > w2 > 0
    assert L.tgl_tcsr_build_workspace(1000, 100, 1) > L.tgl_tcsr_build_workspace(1000, 100, 0) > 0
    assert L.tgl_tcsr_build_workspace(-1, 100, 1) == 0
    assert L.tgl_tcsr_build_workspace(10, 0, 1) == 0
    assert L.tgl_tcsr_build_workspace(10, 10, 2) == 0
    assert L.tgl_tcsr_build_workspace(2**31, 10, 1) == 0             # 2^32 entries
    assert L.tgl_tcsr_build_workspace(2**31 - 1, 10, 1) > 0


FAKE = 0x10000  # a non-null pointer value never dereferenced: every case fails a host check first


def _sample_call(**kw):
    L = P.lib()
    args = dict(g=B.c_tcsr(10, 100, FAKE, FAKE, FAKE, FAKE), roots=FAKE, root_ts=FAKE, n=5, hops=2,
                fan=[10, 10], mode=1, S=1, D=math.inf, ws=FAKE, ws_bytes=1 << 30)
    args.update(kw)
    fa, fp = _fan(args["fan"])
    H = max(len(args["fan"]), 1)
    outs = (B.c_hop_out * H)(*[B.c_hop_out(FAKE, FAKE, FAKE, FAKE, FAKE) for _ in range(H)])
    if "outs" in kw:
        outs = kw["outs"]
    g = args["g"]
    return L.tgl_sample(C.byref(g) if g is not None else None, args["roots"], args["root_ts"],
                        args["n"], args["hops"], fp, args["mode"], args["S"], C.c_float(args["D"]),
                        C.c_uint64(1), C.c_uint64(0), outs, kw.get("counts", FAKE), args["ws"],
                        args["ws_bytes"], None)


@pytest.mark.parametrize("kw", [
    dict(hops=0), dict(hops=9, fan=[1] * 9), dict(fan=[0, 10]), dict(fan=[10, 1025]),
    dict(mode=2), dict(S=0), dict(S=65), dict(S=2, D=math.inf), dict(D=0.0), dict(D=-5.0),
    dict(D=math.nan), dict(n=-1), dict(roots=None), dict(root_ts=None),
    dict(g=B.c_tcsr(0, 100, FAKE, FAKE, FAKE, FAKE)), dict(g=B.c_tcsr(10, 100, None, FAKE, FAKE, FAKE)),
    dict(g=B.c_tcsr(10, 100, FAKE, None, FAKE, FAKE)), dict(g=B.c_tcsr(10, 100, FAKE, FAKE + 8, FAKE, FAKE)),
    dict(g=B.c_tcsr(10, 100, FAKE, FAKE, None, FAKE)), dict(g=B.c_tcsr(10, 100, FAKE, FAKE, FAKE + 4, FAKE)),
    dict(g=B.c_tcsr(10, 100, FAKE, FAKE, FAKE, None)), dict(g=B.c_tcsr(10, 100, FAKE, FAKE, FAKE, FAKE + 8)),
    dict(g=B.c_tcsr(10, 100, FAKE, FAKE, FAKE, FAKE + 64)),
    dict(g=B.c_tcsr(10, 100, FAKE, FAKE, FAKE, FAKE, FAKE + 4)),
    dict(g=B.c_tcsr(10, 100, FAKE, FAKE, FAKE, FAKE, None, FAKE + 4)),           # misaligned histories
    dict(g=B.c_tcsr(10, 100, FAKE, FAKE, FAKE, FAKE, None, None, FAKE + 4)),     # misaligned directory
    dict(g=B.c_tcsr(10, 2**32, FAKE, FAKE, FAKE, FAKE)),
    dict(g=B.c_tcsr(2**31, 100, FAKE, FAKE, FAKE, FAKE)), dict(g=None), dict(counts=None),
])
def test_sample_rejects_invalid_arguments(kw):
    assert _sample_call(**kw) == B.EINVAL


def test_sample_rejects_missing_outputs():
    outs = (B.c_hop_out * 2)(B.c_hop_out(FAKE, FAKE, None, FAKE, None),
                             B.c_hop_out(FAKE, FAKE, FAKE, FAKE, FAKE))
    assert _sample_call(outs=outs) == B.EINVAL
    outs = (B.c_hop_out * 2)(B.c_hop_out(FAKE, FAKE, FAKE, FAKE, None),
                             B.c_hop_out(FAKE, FAKE, FAKE, FAKE, None))   # hop-2 parent missing
    assert _sample_call(outs=outs) == B.EINVAL


def test_sample_workspace_too_small():
    assert _sample_call(ws_bytes=16) == B.ENOSPACE
    assert _sample_call(ws=None) == B.ENOSPACE


def _build_call(**kw):
    L = P.lib()
    a = dict(src=FAKE, dst=FAKE, ts=FAKE, eid=None, m=10, n=5, flags=1, indptr=FAKE,
             ent=FAKE, ts_out=FAKE, nodes=FAKE, tsx=None, hist=None, dir=None, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return L.tgl_tcsr_build(a["src"], a["dst"], a["ts"], a["eid"], a["m"], a["n"], a["flags"],
                            a["indptr"], a["ent"], a["ts_out"], a["nodes"], a["tsx"], a["hist"], a["dir"],
                            a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,want", [
    (dict(m=-1), B.EINVAL), (dict(n=0), B.EINVAL), (dict(n=2**31), B.EINVAL),
    (dict(flags=4), B.EINVAL), (dict(src=None), B.EINVAL), (dict(dst=None), B.EINVAL),
    (dict(ts=None), B.EINVAL), (dict(ent=None), B.EINVAL), (dict(indptr=None), B.EINVAL),
    (dict(ent=FAKE + 4), B.EINVAL), (dict(m=2**31), B.EINVAL),
    (dict(ts_out=None), B.EINVAL), (dict(ts_out=FAKE + 8), B.EINVAL),
    (dict(nodes=None), B.EINVAL), (dict(nodes=FAKE + 4), B.EINVAL), (dict(nodes=FAKE + 64), B.EINVAL), (dict(tsx=FAKE + 8), B.EINVAL),
    (dict(hist=FAKE + 4), B.EINVAL), (dict(dir=FAKE + 4), B.EINVAL),
    (dict(ws_bytes=8), B.ENOSPACE), (dict(ws=None), B.ENOSPACE),
])
def test_build_rejects_invalid_arguments(kw, want):
    assert _build_call(**kw) == want


def test_nodes_rejects_invalid_arguments():
    L = P.lib()
    for args in [(FAKE, FAKE, 0, 10, FAKE), (FAKE, FAKE, 2**31, 10, FAKE), (FAKE, FAKE, 5, -1, FAKE),
                 (FAKE, FAKE, 5, 2**32, FAKE), (None, FAKE, 5, 10, FAKE), (FAKE, None, 5, 10, FAKE),
                 (FAKE, FAKE, 5, 10, None), (FAKE, FAKE, 5, 10, FAKE + 4), (FAKE, FAKE, 5, 10, FAKE + 64)]:
        assert L.tgl_tcsr_nodes(*args, None, None, None, None, None) == B.EINVAL, args
    assert L.tgl_tcsr_nodes(FAKE, FAKE, 5, 10, FAKE, FAKE + 4, None, None, None, None) == B.EINVAL   # misaligned index
    assert L.tgl_tcsr_nodes(FAKE, FAKE, 5, 10, FAKE, None, FAKE + 8, None, None, None) == B.EINVAL   # misaligned entries
    assert L.tgl_tcsr_nodes(FAKE, FAKE, 5, 10, FAKE, None, FAKE, FAKE + 4, None, None) == B.EINVAL   # misaligned histories
    assert L.tgl_tcsr_nodes(FAKE, FAKE, 5, 10, FAKE, None, None, FAKE, None, None) == B.EINVAL   # histories need entries
    assert L.tgl_tcsr_nodes(FAKE, FAKE, 5, 10, FAKE, None, None, None, FAKE + 4, None) == B.EINVAL   # misaligned directory


def test_pack_unpack_reject_invalid_arguments():
    L = P.lib()
    assert L.tgl_tcsr_pack(FAKE, FAKE, None, -1, FAKE, None) == B.EINVAL
    assert L.tgl_tcsr_pack(FAKE, FAKE, None, 2**32, FAKE, None) == B.EINVAL
    assert L.tgl_tcsr_pack(None, FAKE, None, 10, FAKE, None) == B.EINVAL
    assert L.tgl_tcsr_pack(FAKE, None, None, 10, FAKE, None) == B.EINVAL
    assert L.tgl_tcsr_pack(FAKE, FAKE, None, 10, None, None) == B.EINVAL
    assert L.tgl_tcsr_pack(FAKE, FAKE, None, 10, FAKE + 8, None) == B.EINVAL      # misaligned entries
    assert L.tgl_tcsr_unpack(FAKE, -1, FAKE, FAKE, None) == B.EINVAL
    assert L.tgl_tcsr_unpack(FAKE, 2**32, FAKE, FAKE, None) == B.EINVAL
    assert L.tgl_tcsr_unpack(None, 10, FAKE, FAKE, None) == B.EINVAL
    assert L.tgl_tcsr_unpack(FAKE + 4, 10, FAKE, FAKE, None) == B.EINVAL          # misaligned entries


def test_index_len():
    L = P.lib()
    for m, want in [(0, 0), (1, 1), (31, 1), (32, 1), (33, 2), (64, 2), (65, 3), (2**32 - 1, 2**27), (-1, -1)]:
        assert L.tgl_index_len(m) == want, m


def test_timer_argument_checks():
    L = P.lib()
    ms, n = C.c_double(), C.c_int64()
    assert L.tgl_timer_read(7, C.byref(ms), C.byref(n)) == B.EINVAL
    assert L.tgl_timer_read(-1, C.byref(ms), C.byref(n)) == B.EINVAL
    assert L.tgl_timer_read(0, None, C.byref(n)) == B.EINVAL
    assert L.tgl_timer_enable(0) == B.EINVAL
    assert L.tgl_timer_read(0, C.byref(ms), C.byref(n)) == 0 and n.value == 0
    assert L.tgl_timer_select(1 << 7) == B.EINVAL          # no kind 7
    assert L.tgl_timer_select(0x7F) == 0 and L.tgl_timer_select(0) == 0
    P.timer_select()                                        # back to every kind


def _gather_call(n=10, per=1, nt=1, nbr=FAKE, eid=FAKE, count=None, **tab):
    L = P.lib()
    t = dict(rows=FAKE, out=FAKE, num_rows=100, row_bytes=64, key=B.KEY_NODE)
    t.update(tab)
    tabs = (B.c_table * max(nt, 1))(*[B.c_table(t["rows"], t["out"], t["num_rows"], t["row_bytes"], t["key"])
                                      for _ in range(max(nt, 1))])
    return L.tgl_gather(nbr, eid, n, count, per, tabs, nt, None)


@pytest.mark.parametrize("kw", [
    dict(n=-1), dict(per=0), dict(nt=0), dict(nt=9), dict(row_bytes=8), dict(row_bytes=24),
    dict(row_bytes=65552), dict(row_bytes=0), dict(key=2), dict(num_rows=-1), dict(out=None),
    dict(rows=None), dict(rows=FAKE + 8), dict(out=FAKE + 4), dict(nbr=None), dict(key=B.KEY_EDGE, eid=None),
    dict(num_rows=2**62, row_bytes=64),
])
def test_gather_rejects_invalid_arguments(kw):
    assert _gather_call(**kw) == B.EINVAL


def test_gather_empty_is_a_no_op():
    # nothing to gather: valid arguments return OK without touching the device
    assert _gather_call(n=0, out=None) == B.OK
    assert _gather_call(n=0, nbr=None, out=None) == B.OK
    assert _gather_call(n=5, rows=None, num_rows=0, nt=0) == B.EINVAL


def _te_call(dt=FAKE, n=10, count=None, per=1, omega=FAKE, phi=FAKE, dim=100, out_type=B.OUT_F32, out=FAKE):
    return P.lib().tgl_time_encode(dt, n, count, per, omega, phi, dim, out_type, out, None)


@pytest.mark.parametrize("kw", [
    dict(n=-1), dict(per=0), dict(dim=0), dict(dim=4097), dict(out_type=2), dict(omega=None), dict(phi=None),
    dict(dt=None), dict(out=None), dict(out=FAKE + 2), dict(n=2**62, dim=4096),
])
def test_time_encode_rejects_invalid_arguments(kw):
    assert _te_call(**kw) == B.EINVAL


def test_time_encode_empty_is_a_no_op():
    assert _te_call(n=0, dt=None, out=None) == B.OK


def test_sample_ex_rejects_unknown_anchor():
    L = P.lib()
    fa, fp = _fan([10, 10])
    outs = (B.c_hop_out * 2)(*[B.c_hop_out(FAKE, FAKE, FAKE, FAKE, FAKE) for _ in range(2)])
    g = B.c_tcsr(10, 100, FAKE, FAKE, FAKE, FAKE)
    for anchor in (2, -1):
        opts = B.c_sample_opts(anchor, 0)
        assert L.tgl_sample_ex(C.byref(g), FAKE, FAKE, 5, 2, fp, 1, 1, C.c_float(math.inf), C.c_uint64(1),
                               C.c_uint64(0), C.byref(opts), outs, FAKE, FAKE, 1 << 30, None) == B.EINVAL


def test_pointers_reset_rejects_invalid_arguments():
    L = P.lib()
    g = B.c_tcsr(10, 100, FAKE, FAKE, FAKE, FAKE)
    assert L.tgl_pointers_reset(None, 1, FAKE, None) == B.EINVAL
    assert L.tgl_pointers_reset(C.byref(g), 0, FAKE, None) == B.EINVAL
    assert L.tgl_pointers_reset(C.byref(g), 65, FAKE, None) == B.EINVAL
    assert L.tgl_pointers_reset(C.byref(g), 1, None, None) == B.EINVAL
    assert L.tgl_pointers_reset(C.byref(g), 1, FAKE + 2, None) == B.EINVAL
    bad = B.c_tcsr(0, 100, FAKE, FAKE, FAKE, FAKE)
    assert L.tgl_pointers_reset(C.byref(bad), 1, FAKE, None) == B.EINVAL


def test_sample_ex_rejects_misaligned_pointers():
    L = P.lib()
    fa, fp = _fan([10, 10])
    outs = (B.c_hop_out * 2)(*[B.c_hop_out(FAKE, FAKE, FAKE, FAKE, FAKE) for _ in range(2)])
    g = B.c_tcsr(10, 100, FAKE, FAKE, FAKE, FAKE)
    opts = B.c_sample_opts(0, 0, FAKE + 2)
    assert L.tgl_sample_ex(C.byref(g), FAKE, FAKE, 5, 2, fp, 1, 1, C.c_float(math.inf), C.c_uint64(1),
                           C.c_uint64(0), C.byref(opts), outs, FAKE, FAKE, 1 << 30, None) == B.EINVAL


def test_mfg_argument_checks():
    L = P.lib()
    assert L.tgl_mfg_workspace(-1) == 0 and L.tgl_mfg_workspace(10) > 0
    hop = B.c_hop_out(FAKE, FAKE, FAKE, FAKE, FAKE)
    out = B.c_mfg(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)

    def call(hop_=hop, prev=None, roots=FAKE, rts=FAKE, count=FAKE, windows=1, k=10, cap=100, out_=out,
             ws=FAKE, ws_bytes=1 << 30):
        return L.tgl_mfg_export(C.byref(hop_) if hop_ is not None else None,
                                C.byref(prev) if prev is not None else None, roots, rts, count, windows, k, cap,
                                C.byref(out_) if out_ is not None else None, ws, ws_bytes, None)
    for kw in [dict(hop_=None), dict(out_=None), dict(count=None), dict(windows=0), dict(windows=65), dict(k=0),
               dict(k=1025), dict(cap=-1), dict(roots=None), dict(rts=None, roots=FAKE),
               dict(out_=B.c_mfg(FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE)),
               dict(out_=B.c_mfg(None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)),
               dict(hop_=B.c_hop_out(FAKE, None, FAKE, FAKE, FAKE)),
               dict(prev=B.c_hop_out(FAKE, FAKE, FAKE, FAKE, FAKE), windows=2),
               dict(prev=B.c_hop_out(FAKE, FAKE, FAKE, FAKE, FAKE), hop_=B.c_hop_out(FAKE, FAKE, FAKE, FAKE, None))]:
        assert call(**kw) == B.EINVAL, kw
    assert call(ws_bytes=8) == B.ENOSPACE
    assert call(roots=None, rts=None, ws_bytes=8) == B.ENOSPACE   # no roots: accepted up to the workspace
    assert call(ws=None) == B.ENOSPACE


def test_noalloc_argument_checks():
    """tgl_sample_noalloc checks its arguments on the host like tgl_sample,
    and refuses a call whose workspace would exceed its static area."""
    L = P.lib()
    g = B.c_tcsr(10, 100, FAKE, FAKE, FAKE, FAKE)
    outs = (B.c_hop_out * 2)(B.c_hop_out(FAKE, FAKE, FAKE, FAKE, None), B.c_hop_out(FAKE, FAKE, FAKE, FAKE, FAKE))

    def call(n=5, fan=(10, 10), hops=2, mode=1, S=1, delta=float("inf"), gg=g):
        fa, fp = B._i32_array(fan)
        return L.tgl_sample_noalloc(C.byref(gg) if gg is not None else None, FAKE, FAKE, n, hops, fp, mode, S,
                                    C.c_float(delta), 0, 0, outs, FAKE, None)
    assert call(fan=(0, 10)) == B.EINVAL
    assert call(mode=7) == B.EINVAL
    assert call(S=2) == B.EINVAL                     # several snapshots need a finite length
    assert call(gg=None) == B.EINVAL
    assert call(n=20000, fan=(1024, 1024)) == B.ENOSPACE
    need = L.tgl_sample_workspace(20000, 2, B._i32_array((1024, 1024))[1], 1)
    assert need > B.NOALLOC_SCRATCH_BYTES


def test_column_view_binding_checks_its_arguments():
    """tcsr_from_columns refuses columns of the wrong type or length before
    anything reaches the library."""
    import torch
    ip = torch.zeros(3, dtype=torch.int64)
    nbr = torch.zeros(4, dtype=torch.int32)
    ts = torch.zeros(4, dtype=torch.float32)
    eid = torch.zeros(4, dtype=torch.int64)
    for bad in [dict(indptr=ip.int()), dict(nbr=nbr.long()), dict(ts=ts.double()), dict(ts=ts[:3]),
                dict(eid=eid[:3]), dict(eid=eid.int())]:
        a = dict(indptr=ip, nbr=nbr, ts=ts, eid=eid)
        a.update(bad)
        with pytest.raises(ValueError):
            P.tcsr_from_columns(a["indptr"], a["nbr"], a["ts"], a["eid"])
