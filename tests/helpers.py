"""Shared test helpers: golden-file parsing and case decoding (no LoRA arithmetic)."""
import os

import numpy as np

import workloads

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(name):
    """Parse ``key: v1 v2 ...`` lines (``#`` starts a comment) into float64 arrays."""
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, vals = line.split(":", 1)
            out[key.strip()] = np.array([float(v) for v in vals.split()], dtype=np.float64)
    return out


def f64_case(case):
    """Decode a workloads.Case into float64 arrays for the oracle."""
    X = workloads.decode(case.X, case.x_dtype)
    A = [workloads.decode(a, case.w_dtype) if a is not None else None for a in case.A]
    B = [workloads.decode(b, case.w_dtype) if b is not None else None for b in case.B]
    Y = workloads.decode(case.Y, case.y_dtype) if case.Y is not None else None
    dY = workloads.decode(case.dY, case.x_dtype) if case.dY is not None else None
    return X, A, B, Y, dY
