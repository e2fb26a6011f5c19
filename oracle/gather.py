"""Gather/scatter of active blocks (paragraph "Vectorized mixed-schedule
execution": gather extracts each request's active block region into a compact
tensor, scatter writes results back to the corresponding positions).

Test infrastructure: the oracle, not the product path.
"""
from __future__ import annotations

import numpy as np

from .geometry import geometry


def gather_active_blocks(reqs, L: int, dense: np.ndarray):
    """compact[i, j] = dense[row_i, off_i + s_i + j] for j < B_i, zero beyond.
    pos[i, j] = s_i + j (logical position, first prompt token = 0), -1 beyond.
    ``dense`` is [R][W][...] of any dtype."""
    n = len(reqs)
    out = np.zeros((n, L) + dense.shape[2:], dtype=dense.dtype)
    pos = np.full((n, L), -1, dtype=np.int32)
    for i, r in enumerate(reqs):
        q = geometry(r, L)
        for j in range(q.B):
            out[i, j] = dense[q.row, q.off + q.s + j]
            pos[i, j] = q.s + j
    return out, pos


def scatter_active_blocks(reqs, L: int, compact: np.ndarray, dense: np.ndarray) -> np.ndarray:
    """Inverse of the gather: returns a copy of ``dense`` with the active-block
    cells overwritten from ``compact``; every other cell is unchanged."""
    out = dense.copy()
    for i, r in enumerate(reqs):
        q = geometry(r, L)
        for j in range(q.B):
            out[q.row, q.off + q.s + j] = compact[i, j]
    return out
