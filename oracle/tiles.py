"""Tile classes by per-element counting (test infrastructure).

A trace of length L is cut into query tiles of BM rows and key tiles of BN
columns, starting at the trace's first token.  Each tile is EMPTY (0) when
no element ``(i, j)`` with ``i < L``, ``j < L`` and ``j <= i < e_j`` lies in it,
FULL (2) when all BM*BN of its elements are such, and PARTIAL (1) otherwise.
Elements outside the trace count as masked.  The visibility rule is the
eviction mask of Section 2 ("KV-streams").
"""
from __future__ import annotations

import numpy as np

EMPTY, PARTIAL, FULL = 0, 1, 2


def tile_counts(e: np.ndarray, L: int, BM: int, BN: int):
    """Visible-element count per tile, shape [ceil(L/BM), ceil(L/BN)] (int64)."""
    e = np.asarray(e, dtype=np.int64)
    nqt, nkt = -(-L // BM), -(-L // BN)
    i = np.arange(L)[:, None]
    j = np.arange(L)[None, :]
    vis = (j <= i) & (i < np.minimum(e, L)[None, :])
    pad = np.zeros((nqt * BM, nkt * BN), dtype=bool)
    pad[:L, :L] = vis
    return pad.reshape(nqt, BM, nkt, BN).sum(axis=(1, 3))


def tile_classes(e: np.ndarray, L: int, BM: int, BN: int) -> np.ndarray:
    """uint8 class grid of one trace, row-major [ceil(L/BM)][ceil(L/BN)]."""
    c = tile_counts(e, L, BM, BN)
    out = np.full(c.shape, PARTIAL, dtype=np.uint8)
    out[c == 0] = EMPTY
    out[c == BM * BN] = FULL
    return out


def tile_classes_packed(evict_at: np.ndarray, lengths, BM: int, BN: int) -> np.ndarray:
    """Per-trace grids concatenated in trace order (flattened)."""
    parts, off = [], 0
    for L in lengths:
        if L > 0:
            parts.append(tile_classes(evict_at[off:off + L], L, BM, BN).ravel())
        off += L
    return np.concatenate(parts) if parts else np.zeros(0, dtype=np.uint8)
