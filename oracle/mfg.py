"""Oracle for the message-flow-graph block of one sampled hop.

TEST INFRASTRUCTURE ONLY: tests, the smoke check and the benchmark's CPU
baseline leg may use this module; the product library never does.  It shares
no code with the GPU library.

Algorithm 1 ends every layer by generating the MFGs that message passing
runs on.  For one hop the block is fixed by the sampler's output alone:
destination nodes are the hop's groups (hop 1: one per (root, window),
root-major; later hops: one per root), edges are the valid slots in slot
order, and source nodes are the destinations followed by one temporal node
per edge, so edge e runs from source G + e to its group.  A group's valid
slots are the prefix of its k slots before the first PAD.
"""
from __future__ import annotations

import numpy as np


def _prefix_len(nbr2d: np.ndarray) -> np.ndarray:
    pad = nbr2d < 0
    return np.where(pad.any(axis=1), pad.argmax(axis=1), nbr2d.shape[1]).astype(np.int64)


def block(hop, prev, roots, root_ts, windows: int, k: int) -> dict:
    """The block of one hop from the sampler's (oracle's) outputs: ``hop`` and
    ``prev`` carry nbr, eid, ts, dt, parent and num_roots (``prev`` None for
    hop 1)."""
    G = int(hop.num_roots) * windows
    nbr = np.asarray(hop.nbr[:G * k]).reshape(G, k)
    c = _prefix_len(nbr)
    indptr = np.concatenate([[0], np.cumsum(c)]).astype(np.int64)
    mask = np.arange(k)[None, :] < c[:, None]
    if prev is None:
        dst_nid = np.repeat(np.asarray(roots, np.int32), windows)
        dst_ts = np.repeat(np.asarray(root_ts, np.float32), windows)
    else:
        par = np.asarray(hop.parent[:G], np.int64)
        dst_nid = np.asarray(prev.nbr)[par]
        dst_ts = np.asarray(prev.ts)[par]
    return dict(indptr=indptr,
                edge_dst=np.repeat(np.arange(G, dtype=np.int64), c),
                edge_eid=np.asarray(hop.eid[:G * k]).reshape(G, k)[mask],
                edge_dt=np.asarray(hop.dt[:G * k]).reshape(G, k)[mask],
                src_nid=np.concatenate([dst_nid, nbr[mask]]).astype(np.int32),
                src_ts=np.concatenate([dst_ts, np.asarray(hop.ts[:G * k]).reshape(G, k)[mask]]).astype(np.float32),
                G=G, E=int(indptr[-1]))


def block_loop(hop, prev, roots, root_ts, windows: int, k: int) -> dict:
    """The same definition as explicit loops over groups and slots."""
    G = int(hop.num_roots) * windows
    indptr = [0]
    edge_dst, eid, dt, e_nid, e_ts, d_nid, d_ts = [], [], [], [], [], [], []
    for g in range(G):
        if prev is None:
            d_nid.append(int(roots[g // windows]))
            d_ts.append(float(root_ts[g // windows]))
        else:
            p = int(hop.parent[g])
            d_nid.append(int(prev.nbr[p]))
            d_ts.append(float(prev.ts[p]))
        for j in range(k):
            i = g * k + j
            if hop.nbr[i] < 0:
                break
            edge_dst.append(g)
            eid.append(int(hop.eid[i]))
            dt.append(float(hop.dt[i]))
            e_nid.append(int(hop.nbr[i]))
            e_ts.append(float(hop.ts[i]))
        indptr.append(len(edge_dst))
    return dict(indptr=np.array(indptr, np.int64), edge_dst=np.array(edge_dst, np.int64),
                edge_eid=np.array(eid, np.int64), edge_dt=np.array(dt, np.float32),
                src_nid=np.array(d_nid + e_nid, np.int32), src_ts=np.array(d_ts + e_ts, np.float32),
                G=G, E=len(edge_dst))
