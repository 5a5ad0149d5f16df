"""ctypes binding of libtgl (include/tgl.h): argument marshalling only.

Device memory comes from torch tensors and work goes on torch's current
stream; every step of the build and the sampler runs in the HIP library.  If
libtgl.so is missing the first call raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import math
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtgl.so")

OK, EINVAL, ERANGE, ENOSPACE, EDEVICE = 0, -1, -2, -3, -4
MOST_RECENT, UNIFORM = 0, 1
BUILD_UNDIRECTED = 1
MAX_HOPS, MAX_FANOUT, MAX_SNAPSHOTS = 8, 1024, 64
TIMER_HOP1, TIMER_HOPN, TIMER_COMPACT, TIMER_BUILD, TIMER_GATHER, TIMER_TIMEENC, TIMER_MFG = 0, 1, 2, 3, 4, 5, 6
TIMER_KINDS = 7
OUT_F32, OUT_BF16 = 0, 1
KEY_NODE, KEY_EDGE = 0, 1
MAX_TABLES = 8

NODE_WORDS = 32     # int32 words of one node record (128 bytes)
NOALLOC_SCRATCH_BYTES = 128 << 20   # workspace area of tgl_sample_noalloc
NODE_INLINE = 28    # timestamps held inline in a node record
NBR_MASK = 0x7FFFFFFF     # neighbour id bits of a T-CSR entry's nbr field
NBR_FIRST = -0x80000000   # bit 31: the neighbour-first hint (as int32)
INDEX_STRIDE = 32   # entries per sample of the search index

MODES = {"recent": MOST_RECENT, "most_recent": MOST_RECENT, "uniform": UNIFORM,
         MOST_RECENT: MOST_RECENT, UNIFORM: UNIFORM}

# every function declared in include/tgl.h
EXPORTS = ("tgl_version", "tgl_status_str", "tgl_tcsr_build_workspace", "tgl_tcsr_build",
           "tgl_index_len", "tgl_tcsr_nodes", "tgl_tcsr_pack", "tgl_tcsr_unpack", "tgl_sample_capacity", "tgl_sample_workspace", "tgl_sample",
           "tgl_sample_ex", "tgl_sample_noalloc", "tgl_pointers_reset", "tgl_mfg_workspace", "tgl_mfg_export",
           "tgl_gather", "tgl_time_encode", "tgl_timer_enable",
           "tgl_timer_disable", "tgl_timer_read", "tgl_timer_reset", "tgl_timer_select")


class TglError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        super().__init__("%s: %s (%d)" % (what or "libtgl", status_str(status), status))


class c_tcsr(C.Structure):
    _fields_ = [("num_nodes", C.c_int64), ("num_entries", C.c_int64),
                ("indptr", C.c_void_p), ("entries", C.c_void_p), ("ts", C.c_void_p),
                ("nodes", C.c_void_p), ("ts_index", C.c_void_p), ("hist", C.c_void_p),
                ("dir", C.c_void_p)]


class c_table(C.Structure):
    _fields_ = [("rows", C.c_void_p), ("out", C.c_void_p), ("num_rows", C.c_int64),
                ("row_bytes", C.c_int32), ("key", C.c_int32)]


class c_sample_opts(C.Structure):
    _fields_ = [("anchor", C.c_int32), ("reserved", C.c_int32), ("pointers", C.c_void_p)]


ANCHORS = {"own": 0, "root": 1, 0: 0, 1: 1}


class c_mfg(C.Structure):
    _fields_ = [("indptr", C.c_void_p), ("edge_dst", C.c_void_p), ("edge_eid", C.c_void_p),
                ("edge_dt", C.c_void_p), ("src_nid", C.c_void_p), ("src_ts", C.c_void_p),
                ("sizes", C.c_void_p)]


class c_hop_out(C.Structure):
    _fields_ = [("nbr", C.c_void_p), ("eid", C.c_void_p), ("ts", C.c_void_p),
                ("dt", C.c_void_p), ("parent", C.c_void_p)]


_lib: Optional[C.CDLL] = None


def lib() -> C.CDLL:
    """The loaded libtgl.  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libtgl.so not found at %s; build it with "
                           "`python -m paper_2203_14883_amd.build_lib`" % LIB_PATH)
    L = C.CDLL(LIB_PATH)
    P, i32, i64, u32, u64, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_uint64, C.c_float
    L.tgl_version.restype = i32
    L.tgl_version.argtypes = []
    L.tgl_status_str.restype = C.c_char_p
    L.tgl_status_str.argtypes = [i32]
    L.tgl_tcsr_build_workspace.restype = C.c_size_t
    L.tgl_tcsr_build_workspace.argtypes = [i64, i64, u32]
    L.tgl_tcsr_build.restype = i32
    L.tgl_tcsr_build.argtypes = [P, P, P, P, i64, i64, u32, P, P, P, P, P, P, P, P, C.c_size_t, P]
    L.tgl_index_len.restype = i64
    L.tgl_index_len.argtypes = [i64]
    L.tgl_tcsr_nodes.restype = i32
    L.tgl_tcsr_nodes.argtypes = [P, P, i64, i64, P, P, P, P, P, P]
    L.tgl_tcsr_pack.restype = i32
    L.tgl_tcsr_pack.argtypes = [P, P, P, i64, P, P]
    L.tgl_tcsr_unpack.restype = i32
    L.tgl_tcsr_unpack.argtypes = [P, i64, P, P, P]
    L.tgl_sample_capacity.restype = i64
    L.tgl_sample_capacity.argtypes = [i64, i32, P, i32, i32]
    L.tgl_sample_workspace.restype = C.c_size_t
    L.tgl_sample_workspace.argtypes = [i64, i32, P, i32]
    L.tgl_sample.restype = i32
    L.tgl_sample.argtypes = [C.POINTER(c_tcsr), P, P, i64, i32, P, i32, i32, f32, u64, u64,
                             C.POINTER(c_hop_out), P, P, C.c_size_t, P]
    L.tgl_sample_ex.restype = i32
    L.tgl_sample_ex.argtypes = [C.POINTER(c_tcsr), P, P, i64, i32, P, i32, i32, f32, u64, u64,
                                C.POINTER(c_sample_opts), C.POINTER(c_hop_out), P, P, C.c_size_t, P]
    L.tgl_sample_noalloc.restype = i32
    L.tgl_sample_noalloc.argtypes = [C.POINTER(c_tcsr), P, P, i64, i32, P, i32, i32, f32, u64, u64,
                                     C.POINTER(c_hop_out), P, P]
    L.tgl_pointers_reset.restype = i32
    L.tgl_pointers_reset.argtypes = [C.POINTER(c_tcsr), i32, P, P]
    L.tgl_mfg_workspace.restype = C.c_size_t
    L.tgl_mfg_workspace.argtypes = [i64]
    L.tgl_mfg_export.restype = i32
    L.tgl_mfg_export.argtypes = [C.POINTER(c_hop_out), C.POINTER(c_hop_out), P, P, P, i32, i32, i64,
                                 C.POINTER(c_mfg), P, C.c_size_t, P]
    L.tgl_gather.restype = i32
    L.tgl_gather.argtypes = [P, P, i64, P, i64, C.POINTER(c_table), i32, P]
    L.tgl_time_encode.restype = i32
    L.tgl_time_encode.argtypes = [P, i64, P, i64, P, P, i32, i32, P, P]
    L.tgl_timer_enable.restype = i32
    L.tgl_timer_enable.argtypes = [i32]
    L.tgl_timer_disable.restype = i32
    L.tgl_timer_disable.argtypes = []
    L.tgl_timer_reset.restype = i32
    L.tgl_timer_reset.argtypes = []
    L.tgl_timer_read.restype = i32
    L.tgl_timer_read.argtypes = [i32, C.POINTER(C.c_double), C.POINTER(C.c_int64)]
    L.tgl_timer_select.restype = i32
    L.tgl_timer_select.argtypes = [C.c_uint32]
    _lib = L
    return L


def status_str(s: int) -> str:
    return lib().tgl_status_str(int(s)).decode()


def _check(s: int, what: str):
    if s != OK:
        raise TglError(int(s), what)


def _p(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _i32_array(v: Sequence[int]):
    a = np.ascontiguousarray(np.asarray(v, dtype=np.int32))
    return a, a.ctypes.data_as(C.c_void_p)


# --------------------------------------------------------------------------
# T-CSR
# --------------------------------------------------------------------------

@dataclass
class TCSR:
    """Device T-CSR: indptr int64[N+1]; entries int64[M, 2] holding the 16-byte
    records (int32 nbr, float32 ts | int64 eid), bit 31 of nbr being the
    neighbour-first hint (set: the neighbour has no entry below this entry's
    ts); ts float32[M], the entries' timestamps as the separate search array; nodes int32[N, 32], the per-node
    128-byte records (uint32 start, uint32 end, float32 first ts, float32 last
    ts, then float32 ts of the run's first 28 entries, +inf beyond);
    ts_index float32[ceil(M / 32)], every 32nd timestamp (the search index), or
    None; hist int32[M, 2], per entry the positions [lo, hi) of the neighbour's
    entries older than it (the neighbour's history), or None; dir int32[ceil(M /
    32), 2], the runs' time directories (per search-index slot, a cell's first
    position and its timestamp's float32 bits), or None."""
    indptr: torch.Tensor
    entries: torch.Tensor
    ts: torch.Tensor
    nodes: torch.Tensor
    num_nodes: int
    ts_index: Optional[torch.Tensor] = None
    hist: Optional[torch.Tensor] = None
    dir: Optional[torch.Tensor] = None

    @property
    def num_entries(self) -> int:
        return int(self.entries.shape[0])

    @property
    def nbr(self) -> torch.Tensor:
        """Neighbour ids (the hint bit cleared)."""
        return self.entries.view(torch.int32)[:, 0] & NBR_MASK

    @property
    def first_hint(self) -> torch.Tensor:
        """Per entry: the neighbour-first hint bit."""
        return self.entries.view(torch.int32)[:, 0] < 0

    @property
    def entry_ts(self) -> torch.Tensor:
        return self.entries.view(torch.float32)[:, 1]

    @property
    def eid(self) -> torch.Tensor:
        return self.entries[:, 1]

    def c_view(self) -> c_tcsr:
        m = self.num_entries
        return c_tcsr(self.num_nodes, m, self.indptr.data_ptr(),
                      self.entries.data_ptr() if m else None, self.ts.data_ptr() if m else None,
                      self.nodes.data_ptr(),
                      self.ts_index.data_ptr() if m and self.ts_index is not None else None,
                      self.hist.data_ptr() if m and self.hist is not None else None,
                      self.dir.data_ptr() if m and self.dir is not None else None)


def pack_entries(nbr: np.ndarray, ts: np.ndarray, eid: np.ndarray) -> np.ndarray:
    """Host-side packing of structure-of-arrays T-CSR fields into records."""
    m = len(nbr)
    rec = np.zeros((m, 4), dtype=np.int32)
    rec[:, 0] = np.asarray(nbr, np.int32)
    rec[:, 1] = np.asarray(ts, np.float32).view(np.int32)
    rec.view(np.int64)[:, 1] = np.asarray(eid, np.int64)
    return rec.view(np.int64).reshape(m, 2)


def index_len(num_entries: int) -> int:
    return int(lib().tgl_index_len(int(num_entries)))


def tcsr_from_host(indptr, nbr, ts, eid, device="cuda", index: bool = True, hints: bool = True,
                   hist: bool = True, dir: bool = True) -> TCSR:
    """Uploads a T-CSR given as host arrays (e.g. one built elsewhere) and
    computes its node summaries, if `index` its search index, if `hints` the
    neighbour-first hint bits (else they stay clear), if `hist` the
    neighbour histories and if `dir` the time directories."""
    rec = pack_entries(nbr, ts, eid)
    ent = torch.from_numpy(rec).to(device)
    tsa = torch.from_numpy(np.ascontiguousarray(np.asarray(ts, np.float32))).to(device)
    if ent.shape[0] == 0:
        ent = torch.empty((0, 2), dtype=torch.int64, device=device)
        tsa = torch.empty(0, dtype=torch.float32, device=device)
    n = len(indptr) - 1
    ip = torch.from_numpy(np.asarray(indptr, np.int64)).to(device)
    nodes = torch.empty((n, NODE_WORDS), dtype=torch.int32, device=device)
    m = int(ent.shape[0])
    tsx = torch.empty(index_len(m), dtype=torch.float32, device=device) if index else None
    hs = torch.empty((m, 2), dtype=torch.int32, device=device) if hist else None
    td = torch.empty((index_len(m), 2), dtype=torch.int32, device=device) if dir else None
    _check(lib().tgl_tcsr_nodes(_p(ip), _p(tsa) if m else None, n, m, _p(nodes),
                                _p(tsx) if index and m else None, _p(ent) if (hints or hist) and m else None,
                                _p(hs) if hist and m else None, _p(td) if dir and m else None, _stream()),
           "tgl_tcsr_nodes")
    if hist and not hints and m:
        ent.view(torch.int32)[:, 0] &= NBR_MASK     # histories need the entries; keep the hint bits clear
    return TCSR(ip, ent, tsa, nodes, n, tsx, hs, td)


def tcsr_from_columns(indptr: torch.Tensor, nbr: torch.Tensor, ts: torch.Tensor, eid: Optional[torch.Tensor],
                      index: bool = True, hints: bool = True, hist: bool = True, dir: bool = True,
                      stream=None) -> TCSR:
    """A T-CSR from device columns (int64 indptr[N+1], int32 nbr, float32 ts,
    int64 eid or None for eid = position), packed into entries on the device,
    with its node records and, as asked, search index, hints, histories and
    time directories.  `ts` becomes the T-CSR's timestamp array."""
    m = int(nbr.shape[0])
    for t, dt in ((indptr, torch.int64), (nbr, torch.int32), (ts, torch.float32)):
        if t.dtype != dt or not t.is_contiguous():
            raise ValueError("indptr must be int64, nbr int32, ts float32, all contiguous")
    if ts.shape[0] != m or (eid is not None and (eid.dtype != torch.int64 or not eid.is_contiguous()
                                                   or eid.shape[0] != m)):
        raise ValueError("nbr, ts and eid must have the same length")
    dev = nbr.device
    n = int(indptr.shape[0]) - 1
    ent = torch.empty((m, 2), dtype=torch.int64, device=dev)
    st = _stream(stream)
    _check(lib().tgl_tcsr_pack(_p(nbr) if m else None, _p(ts) if m else None, _p(eid) if m else None, m,
                               _p(ent) if m else None, st), "tgl_tcsr_pack")
    nodes = torch.empty((n, NODE_WORDS), dtype=torch.int32, device=dev)
    tsx = torch.empty(index_len(m), dtype=torch.float32, device=dev) if index else None
    hs = torch.empty((m, 2), dtype=torch.int32, device=dev) if hist else None
    td = torch.empty((index_len(m), 2), dtype=torch.int32, device=dev) if dir else None
    _check(lib().tgl_tcsr_nodes(_p(indptr), _p(ts) if m else None, n, m, _p(nodes),
                                _p(tsx) if index and m else None, _p(ent) if (hints or hist) and m else None,
                                _p(hs) if hist and m else None, _p(td) if dir and m else None, st),
           "tgl_tcsr_nodes")
    if hist and not hints and m:
        ent.view(torch.int32)[:, 0] &= NBR_MASK
    return TCSR(indptr, ent, ts, nodes, n, tsx, hs, td)


def tcsr_columns(g: TCSR, stream=None):
    """The neighbour ids (hint bits cleared) and edge ids of a device T-CSR's
    entries as separate int32 and int64 columns, unpacked on the device."""
    m = g.num_entries
    nbr = torch.empty(m, dtype=torch.int32, device=g.entries.device)
    eid = torch.empty(m, dtype=torch.int64, device=g.entries.device)
    _check(lib().tgl_tcsr_unpack(_p(g.entries) if m else None, m, _p(nbr) if m else None,
                                 _p(eid) if m else None, _stream(stream)), "tgl_tcsr_unpack")
    return nbr, eid


def tcsr_build_workspace(num_edges: int, num_nodes: int, undirected: bool = True) -> int:
    return int(lib().tgl_tcsr_build_workspace(num_edges, num_nodes,
                                              BUILD_UNDIRECTED if undirected else 0))


def tcsr_build(src: torch.Tensor, dst: torch.Tensor, ts: torch.Tensor,
               eid: Optional[torch.Tensor], num_nodes: int, undirected: bool = True,
               workspace: Optional[torch.Tensor] = None, stream=None, index: bool = True,
               hist: bool = True, dir: bool = True) -> TCSR:
    """Builds the T-CSR of a device COO (int32 src/dst, float32 ts, int64 eid or
    None), with its search index if `index`, its neighbour histories if
    `hist` and its time directories if `dir`."""
    L = lib()
    m0 = int(src.shape[0])
    flags = BUILD_UNDIRECTED if undirected else 0
    for t, dt in ((src, torch.int32), (dst, torch.int32), (ts, torch.float32)):
        if t.dtype != dt or not t.is_contiguous() or t.shape[0] != m0:
            raise ValueError("src/dst must be int32, ts float32, contiguous, same length")
    if eid is not None and (eid.dtype != torch.int64 or not eid.is_contiguous() or eid.shape[0] != m0):
        raise ValueError("eid must be a contiguous int64 tensor of the same length")
    M = 2 * m0 if undirected else m0
    dev = src.device
    indptr = torch.empty(num_nodes + 1, dtype=torch.int64, device=dev)
    entries = torch.empty((M, 2), dtype=torch.int64, device=dev)
    tsa = torch.empty(M, dtype=torch.float32, device=dev)
    nodes = torch.empty((num_nodes, NODE_WORDS), dtype=torch.int32, device=dev)
    tsx = torch.empty(index_len(M), dtype=torch.float32, device=dev) if index else None
    hs = torch.empty((M, 2), dtype=torch.int32, device=dev) if hist else None
    td = torch.empty((index_len(M), 2), dtype=torch.int32, device=dev) if dir else None
    need = int(L.tgl_tcsr_build_workspace(m0, num_nodes, flags))
    if need == 0:
        raise TglError(EINVAL, "tgl_tcsr_build_workspace")
    own_ws = workspace is None
    if own_ws:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    s = L.tgl_tcsr_build(_p(src), _p(dst), _p(ts), _p(eid), m0, num_nodes, flags, _p(indptr),
                         _p(entries) if M else None, _p(tsa) if M else None, _p(nodes),
                         _p(tsx) if index and M else None, _p(hs) if hist and M else None,
                         _p(td) if dir and M else None, _p(workspace), workspace.numel(), _stream(stream))
    if own_ws:
        del workspace
    _check(s, "tgl_tcsr_build")
    return TCSR(indptr, entries, tsa, nodes, num_nodes, tsx, hs, td)


# --------------------------------------------------------------------------
# sampler
# --------------------------------------------------------------------------

@dataclass
class Hop:
    nbr: torch.Tensor
    eid: torch.Tensor
    ts: torch.Tensor
    dt: torch.Tensor
    parent: Optional[torch.Tensor]
    num_roots: int


def sample_capacity(num_roots: int, fanouts: Sequence[int], snapshots: int, hop: int) -> int:
    fa, fp = _i32_array(fanouts)
    return int(lib().tgl_sample_capacity(num_roots, len(fa), fp, snapshots, hop))


class Sampler:
    """Preallocated outputs and workspace for repeated calls with up to
    ``max_roots`` roots and fixed fanouts / snapshots.  ``run`` enqueues one
    call and returns without synchronising; ``hops`` slices the results."""

    def __init__(self, max_roots: int, fanouts: Sequence[int], snapshots: int = 1,
                 device="cuda"):
        L = lib()
        self.fanouts = tuple(int(k) for k in fanouts)
        self.snapshots = int(snapshots)
        self.max_roots = int(max_roots)
        self._fa, self._fp = _i32_array(self.fanouts)
        H = len(self.fanouts)
        caps = [int(L.tgl_sample_capacity(self.max_roots, H, self._fp, self.snapshots, h))
                for h in range(H + 1)]
        if min(caps) < 0:
            raise TglError(EINVAL, "tgl_sample_capacity")
        self.caps = caps
        dev = torch.device(device)
        self.nbr = [torch.empty(max(caps[h + 1], 1), dtype=torch.int32, device=dev) for h in range(H)]
        self.eid = [torch.empty(max(caps[h + 1], 1), dtype=torch.int64, device=dev) for h in range(H)]
        self.ts = [torch.empty(max(caps[h + 1], 1), dtype=torch.float32, device=dev) for h in range(H)]
        self.dt = [torch.empty(max(caps[h + 1], 1), dtype=torch.float32, device=dev) for h in range(H)]
        self.parent = [None] + [torch.empty(max(caps[h], 1), dtype=torch.int64, device=dev)
                                for h in range(1, H)]
        self.counts = torch.zeros(H, dtype=torch.int64, device=dev)
        ws = int(L.tgl_sample_workspace(self.max_roots, H, self._fp, self.snapshots))
        self.workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=dev)
        outs = (c_hop_out * H)()
        for h in range(H):
            outs[h] = c_hop_out(self.nbr[h].data_ptr(), self.eid[h].data_ptr(), self.ts[h].data_ptr(),
                                self.dt[h].data_ptr(),
                                None if self.parent[h] is None else self.parent[h].data_ptr())
        self._outs = outs

    def run(self, g: TCSR, roots: torch.Tensor, root_ts: torch.Tensor, mode="uniform",
            snapshot_len: float = math.inf, seed: int = 0, root_base: int = 0, stream=None,
            num_roots: Optional[int] = None, anchor="own", pointers: Optional[torch.Tensor] = None):
        """Enqueues one sampling call.  ``anchor`` places the snapshot windows
        of hops >= 2 at the root's own time ("own") or at its hop-1 ancestor's
        time, cut below its own ("root").  ``pointers`` (from
        ``pointers_reset``) makes hop 1 start from, and advance, saved window
        edges (Sec. 3.1); the samples are the same."""
        n = int(roots.shape[0]) if num_roots is None else int(num_roots)
        if n > self.max_roots:
            raise ValueError("more roots than the sampler was sized for")
        if roots.dtype != torch.int32 or root_ts.dtype != torch.float32:
            raise ValueError("roots must be int32 and root_ts float32")
        if not roots.is_contiguous() or not root_ts.is_contiguous():
            raise ValueError("roots and root_ts must be contiguous")
        view = g.c_view()
        if pointers is not None and (pointers.dtype != torch.int32 or not pointers.is_contiguous()
                                     or pointers.numel() != (self.snapshots + 1) * g.num_nodes):
            raise ValueError("pointers must be a contiguous int32 tensor of (snapshots + 1) * num_nodes")
        opts = c_sample_opts(ANCHORS[anchor], 0, None if pointers is None else pointers.data_ptr())
        s = lib().tgl_sample_ex(C.byref(view), _p(roots), _p(root_ts), n, len(self.fanouts), self._fp,
                                MODES[mode], self.snapshots, C.c_float(snapshot_len),
                                C.c_uint64(seed & (2**64 - 1)), C.c_uint64(root_base & (2**64 - 1)),
                                C.byref(opts), self._outs, _p(self.counts), _p(self.workspace),
                                self.workspace.numel(), _stream(stream))
        _check(s, "tgl_sample_ex")

    def hops(self) -> List[Hop]:
        """Slices the outputs of the last call by the per-hop root counts (syncs)."""
        counts = self.counts.cpu().tolist()
        out = []
        for h, k in enumerate(self.fanouts):
            nr = int(counts[h])
            n = nr * (self.snapshots if h == 0 else 1) * k
            out.append(Hop(self.nbr[h][:n], self.eid[h][:n], self.ts[h][:n], self.dt[h][:n],
                           None if h == 0 else self.parent[h][:nr], nr))
        return out


@dataclass
class MFG:
    """One hop's block (Alg. 1, "generate DGL MFGs") in CSC form, at capacity:
    the first G + 1 entries of ``indptr``, E of the edge arrays and G + E of
    the source arrays are valid, with (G, E) in the device tensor ``sizes``.
    Edge e runs from source node G + e to destination group ``edge_dst[e]``;
    source nodes 0..G-1 are the destination groups themselves."""
    indptr: torch.Tensor
    edge_dst: torch.Tensor
    edge_eid: torch.Tensor
    edge_dt: torch.Tensor
    src_nid: torch.Tensor
    src_ts: torch.Tensor
    sizes: torch.Tensor

    def sliced(self) -> "MFG":
        """The valid parts (synchronises to read the sizes)."""
        G, E = (int(v) for v in self.sizes.cpu().tolist())
        return MFG(self.indptr[:G + 1], self.edge_dst[:E], self.edge_eid[:E], self.edge_dt[:E],
                   self.src_nid[:G + E], self.src_ts[:G + E], self.sizes)


def mfg_export(smp: "Sampler", h: int, roots: torch.Tensor, root_ts: torch.Tensor, stream=None) -> MFG:
    """Block of hop ``h`` (0-based) of the sampler's last call, built on the
    device from its outputs without synchronising."""
    L = lib()
    windows = smp.snapshots if h == 0 else 1
    k = smp.fanouts[h]
    gcap = smp.caps[h] * windows
    dev = smp.counts.device
    m = MFG(torch.empty(gcap + 1, dtype=torch.int64, device=dev),
            torch.empty(max(gcap * k, 1), dtype=torch.int64, device=dev),
            torch.empty(max(gcap * k, 1), dtype=torch.int64, device=dev),
            torch.empty(max(gcap * k, 1), dtype=torch.float32, device=dev),
            torch.empty(max(gcap * (k + 1), 1), dtype=torch.int32, device=dev),
            torch.empty(max(gcap * (k + 1), 1), dtype=torch.float32, device=dev),
            torch.zeros(2, dtype=torch.int64, device=dev))
    ws_bytes = int(L.tgl_mfg_workspace(gcap))
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    out = c_mfg(m.indptr.data_ptr(), m.edge_dst.data_ptr(), m.edge_eid.data_ptr(), m.edge_dt.data_ptr(),
                m.src_nid.data_ptr(), m.src_ts.data_ptr(), m.sizes.data_ptr())
    prev = C.byref(smp._outs[h - 1]) if h > 0 else None
    s = L.tgl_mfg_export(C.byref(smp._outs[h]), prev, _p(roots), _p(root_ts),
                         smp.counts.data_ptr() + 8 * h, windows, k, gcap, C.byref(out), _p(ws), ws.numel(),
                         _stream(stream))
    _check(s, "tgl_mfg_export")
    m._ws = ws          # keep the workspace alive until the stream has used it
    return m


def pointers_reset(g: TCSR, snapshots: int = 1, pointers: Optional[torch.Tensor] = None,
                   stream=None) -> torch.Tensor:
    """Saved window edges of hop 1 (Sec. 3.1's per-node pointers), one per node
    and window edge, set to the start of every run; allocated here unless
    given.  Stored as int32 (the library reads them as uint32 positions)."""
    n = (int(snapshots) + 1) * g.num_nodes
    if pointers is None:
        pointers = torch.empty(n, dtype=torch.int32, device=g.indptr.device)
    view = g.c_view()
    _check(lib().tgl_pointers_reset(C.byref(view), int(snapshots), pointers.data_ptr(), _stream(stream)),
           "tgl_pointers_reset")
    return pointers


def sample(g: TCSR, roots: torch.Tensor, root_ts: torch.Tensor, fanouts: Sequence[int],
           mode="uniform", snapshots: int = 1, snapshot_len: float = math.inf, seed: int = 0,
           root_base: int = 0, stream=None, anchor="own") -> List[Hop]:
    """One-shot sampling call; returns per-hop outputs sliced to their sizes."""
    smp = Sampler(max(int(roots.shape[0]), 0), fanouts, snapshots, device=roots.device)
    smp.run(g, roots, root_ts, mode, snapshot_len, seed, root_base, stream, anchor=anchor)
    return smp.hops()


# --------------------------------------------------------------------------
# feature / state gather
# --------------------------------------------------------------------------

KEYS = {"node": KEY_NODE, "edge": KEY_EDGE, KEY_NODE: KEY_NODE, KEY_EDGE: KEY_EDGE}


def _row_bytes(t: torch.Tensor) -> int:
    if t.dim() < 1 or not t.is_contiguous():
        raise ValueError("a table must be a contiguous tensor of rows")
    return int(t[0].numel() * t.element_size()) if t.shape[0] else int(
        math.prod(t.shape[1:]) * t.element_size())


def gather(nbr: Optional[torch.Tensor], eid: Optional[torch.Tensor], tables, n: Optional[int] = None,
           count: Optional[torch.Tensor] = None, per_count: int = 1, outs=None, stream=None):
    """Looks up one row per slot in each table (Fig. 2, steps 2-3).

    ``tables`` is a list of ``(rows, key)`` with ``rows`` a contiguous
    ``[num_rows, ...]`` tensor (row size a multiple of 16 bytes) and ``key``
    ``"node"`` (rows indexed by ``nbr``) or ``"edge"`` (by ``eid``).  Slot i of
    the output of a table is ``rows[key_i]``, or zeros when the key is outside
    ``[0, num_rows)`` (PAD slots carry -1).  With ``count`` (a device int64
    tensor) only slots ``i < min(n, count[0] * per_count)`` are written.
    Returns the outputs (allocated here unless ``outs`` is given)."""
    if n is None:
        ref = nbr if nbr is not None else eid
        n = int(ref.shape[0])
    if nbr is not None and (nbr.dtype != torch.int32 or not nbr.is_contiguous()):
        raise ValueError("nbr must be a contiguous int32 tensor")
    if eid is not None and (eid.dtype != torch.int64 or not eid.is_contiguous()):
        raise ValueError("eid must be a contiguous int64 tensor")
    if count is not None and (count.dtype != torch.int64 or count.device.type != "cuda"):
        raise ValueError("count must be a device int64 tensor")
    tabs = (c_table * max(len(tables), 1))()
    result = []
    for i, (rows, key) in enumerate(tables):
        rb = _row_bytes(rows)
        out = outs[i] if outs is not None else torch.empty((n,) + tuple(rows.shape[1:]), dtype=rows.dtype,
                                                            device=rows.device)
        tabs[i] = c_table(rows.data_ptr() if rows.numel() else None, out.data_ptr() if n else None,
                          int(rows.shape[0]), rb, KEYS[key])
        result.append(out)
    s = lib().tgl_gather(_p(nbr), _p(eid), int(n), _p(count), int(per_count), tabs, len(tables),
                         _stream(stream))
    _check(s, "tgl_gather")
    return result


# --------------------------------------------------------------------------
# time encoding (Eq. 3)
# --------------------------------------------------------------------------

def time_encode(dt: torch.Tensor, omega: torch.Tensor, phi: torch.Tensor, out_dtype=torch.float32,
                n: Optional[int] = None, count: Optional[torch.Tensor] = None, per_count: int = 1,
                out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Row i = cos(omega * dt[i] + phi) for dt[i] >= 0, zeros for PAD slots
    (dt = -1); ``[n, dim]`` float32 or bfloat16.  With ``count`` (a device
    int64 tensor) only rows ``i < min(n, count[0] * per_count)`` are written."""
    if dt.dtype != torch.float32 or not dt.is_contiguous():
        raise ValueError("dt must be a contiguous float32 tensor")
    for t in (omega, phi):
        if t.dtype != torch.float32 or not t.is_contiguous() or t.dim() != 1:
            raise ValueError("omega and phi must be contiguous float32 vectors")
    if omega.numel() != phi.numel():
        raise ValueError("omega and phi must have the same length")
    if out_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out_dtype must be float32 or bfloat16")
    if count is not None and (count.dtype != torch.int64 or count.device.type != "cuda"):
        raise ValueError("count must be a device int64 tensor")
    n = int(dt.shape[0]) if n is None else int(n)
    dim = int(omega.numel())
    if out is None:
        out = torch.empty((n, dim), dtype=out_dtype, device=dt.device)
    s = lib().tgl_time_encode(_p(dt), n, _p(count), int(per_count), _p(omega), _p(phi), dim,
                              OUT_F32 if out_dtype == torch.float32 else OUT_BF16,
                              out.data_ptr() if n else None, _stream(stream))
    _check(s, "tgl_time_encode")
    return out


# --------------------------------------------------------------------------
# kernel timers
# --------------------------------------------------------------------------

def timer_enable(capacity: int = 4096):
    _check(lib().tgl_timer_enable(capacity), "tgl_timer_enable")


def timer_disable():
    _check(lib().tgl_timer_disable(), "tgl_timer_disable")


def timer_reset():
    _check(lib().tgl_timer_reset(), "tgl_timer_reset")


def timer_select(*kinds: int):
    """Record only launches of the given timer kinds (none given: all)."""
    mask = 0
    for k in kinds:
        mask |= 1 << int(k)
    _check(lib().tgl_timer_select(mask if kinds else (1 << TIMER_KINDS) - 1), "tgl_timer_select")


def timer_read(kind: int):
    ms = C.c_double()
    n = C.c_int64()
    _check(lib().tgl_timer_read(kind, C.byref(ms), C.byref(n)), "tgl_timer_read")
    return ms.value, n.value
