"""Reader for the hand-worked fixtures under tests/golden/."""
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read(name):
    """Parse "key: values" lines; a key ending in ".slots:" collects the
    following lines (one slot "nbr eid ts dt" each) until a blank line."""
    out, key = {}, None
    with open(os.path.join(GOLDEN, name)) as f:
        for raw in f:
            line = raw.split("#", 1)[0].rstrip()
            if key is not None:
                if not line.strip():
                    key = None
                    continue
                out[key].append([float(v) for v in line.split()])
                continue
            if not line.strip():
                continue
            k, _, v = line.partition(":")
            k = k.strip()
            if k.endswith(".slots"):
                out[k] = []
                key = k
            else:
                out[k] = v.split()
    return out


def ints(v):
    return np.array([int(x) for x in v], dtype=np.int64)


def floats(v):
    return np.array([math.inf if x == "inf" else float(x) for x in v], dtype=np.float64)
