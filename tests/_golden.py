"""Reader for the small text fixtures under tests/golden/."""
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name):
    """Parse 'key v1 v2 ...' lines; '#' starts a comment line."""
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            out[key] = vals
    return out


def f32(vals):
    return np.array([float(v) for v in vals], dtype=np.float32)


def i32(vals):
    return np.array([int(v) for v in vals], dtype=np.int32)
