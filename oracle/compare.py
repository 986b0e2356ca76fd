"""Error metric of the parity tests (oracle side; test infrastructure only).

For a state or gradient tensor T against the fp64 reference R, rows r:

    rel = max_r ||T_r - R_r||_inf / max(||R_r||_inf, 1e-3 * ||R||_inf)

so that every row is judged against its own scale, with a floor that keeps
rows of (near) zero reference from dividing by zero.  Weight gradients are
compared as one row (``whole=True``).  The paper fixes no metric; this one
is the reading the tests use.
"""
from __future__ import annotations

import numpy as np


def rel_err(T, R, whole: bool = False) -> float:
    T = np.asarray(T, dtype=np.float64)
    R = np.asarray(R, dtype=np.float64)
    if T.shape != R.shape:
        raise ValueError(f"shape mismatch {T.shape} vs {R.shape}")
    if R.size == 0:
        return 0.0
    if whole or R.ndim == 1:
        T = T.reshape(1, -1)
        R = R.reshape(1, -1)
    else:
        T = T.reshape(R.shape[0], -1)
        R = R.reshape(R.shape[0], -1)
    scale = np.abs(R).max()
    if scale == 0.0:
        return float(np.abs(T).max())
    row_ref = np.maximum(np.abs(R).max(axis=1), 1e-3 * scale)
    return float((np.abs(T - R).max(axis=1) / row_ref).max())
