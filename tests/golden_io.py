"""Reader for the hand-derived fixtures under tests/golden/."""
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, val = line.split(":", 1)
            if "|" in val:
                shape, vals = val.split("|")
                shape = tuple(int(v) for v in shape.split())
                arr = np.array([float(v) for v in vals.split()], dtype=np.float64)
                out[key.strip()] = arr.reshape(shape)
            else:
                out[key.strip()] = float(val)
    return out
