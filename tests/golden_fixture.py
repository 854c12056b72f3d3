"""Reader of tests/golden/algorithm1_worked_example.txt (test infrastructure)."""
import os

import numpy as np

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "algorithm1_worked_example.txt")

INT_KEYS = {"n_total", "world", "worker", "union_own_first"}


def load():
    """The fixture as a dict: scalars as int/float, lists as numpy arrays
    (int32 for index lists, float32 for values)."""
    out = {}
    for line in open(PATH):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, val = line.split(":", 1)
        key = key.strip()
        parts = val.split()
        if key in INT_KEYS or key.startswith("cycle_"):
            out[key] = int(parts[0])
        elif key.startswith("idx_") or key == "union":
            out[key] = np.array([int(p) for p in parts], np.int32)
        elif len(parts) == 1 and not key.startswith(("val_", "grad_", "residual_", "union_")):
            out[key] = float(parts[0])
        else:
            out[key] = np.array([float(p) for p in parts], np.float32)
    return out
