"""Oracle for what the sampled slots feed: the lookup of per-node and
per-edge rows, and the time encoding of the slots' time differences.

TEST INFRASTRUCTURE ONLY: tests, the smoke check and the benchmark's CPU
baseline leg may use this module; the product library never does.  It shares
no code with the GPU library.

Figure 2 of TGL (steps 2 and 3) fetches, for the nodes and edges of a sampled
mini-batch, their node features, node memory and mailbox rows (by node id)
and their edge features (by edge id); Table 3 lists the row widths.  The
lookup has a plain definition: output row i of a table is the table's row
``key_i``, where ``key_i`` is the slot's neighbour id or edge id.  A padded
slot (key -1) has no node or edge; it gets a row of zeros, as does any key
outside the table.

Equation 3 (the time encoder of Section 2) maps a time difference dt to
cos(omega * dt + phi); ``time_encode`` evaluates it per slot in float64.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np

NODE, EDGE = "node", "edge"


def gather(nbr: Optional[np.ndarray], eid: Optional[np.ndarray],
           tables: Sequence[Tuple[np.ndarray, str]], limit: Optional[int] = None) -> List[np.ndarray]:
    """out[t][i] = tables[t].rows[key_i] for key_i in [0, num_rows), zeros
    otherwise, for i < limit (default: every slot).  ``key_i`` is ``nbr[i]``
    for a table keyed by node and ``eid[i]`` for one keyed by edge."""
    outs = []
    for rows, key in tables:
        keys = np.asarray(nbr if key == NODE else eid, dtype=np.int64)
        n = len(keys) if limit is None else max(0, min(int(limit), len(keys)))
        keys = keys[:n]
        out = np.zeros((n,) + rows.shape[1:], dtype=rows.dtype)
        ok = (keys >= 0) & (keys < rows.shape[0])
        out[ok] = rows[keys[ok]]
        outs.append(out)
    return outs


def gather_loop(nbr, eid, tables, limit=None):
    """The same definition as an explicit loop over slots (for tiny inputs)."""
    outs = []
    for rows, key in tables:
        keys = nbr if key == NODE else eid
        n = len(keys) if limit is None else max(0, min(int(limit), len(keys)))
        out = []
        for i in range(n):
            k = int(keys[i])
            out.append(rows[k].copy() if 0 <= k < rows.shape[0] else np.zeros(rows.shape[1:], rows.dtype))
        outs.append(np.array(out, dtype=rows.dtype).reshape((n,) + rows.shape[1:]))
    return outs


def time_encode(dt: np.ndarray, omega: np.ndarray, phi: np.ndarray, limit: Optional[int] = None) -> np.ndarray:
    """Equation 3 (the time encoder of Section 2): row i is
    cos(omega * dt[i] + phi) for a slot with dt[i] >= 0 and zeros for a padded
    slot (dt = -1), for i < limit (default: every slot).  Evaluated in float64
    from the float32 inputs: the product of two float32 values is exact in
    float64, so the only roundings are the sum's and the cosine's."""
    dt = np.asarray(dt, np.float32)
    n = len(dt) if limit is None else max(0, min(int(limit), len(dt)))
    d = dt[:n].astype(np.float64)[:, None]
    w = np.asarray(omega, np.float32).astype(np.float64)[None, :]
    p = np.asarray(phi, np.float32).astype(np.float64)[None, :]
    out = np.cos(d * w + p)
    out[~(d[:, 0] >= 0.0)] = 0.0
    return out
