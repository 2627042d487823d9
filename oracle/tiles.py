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


def tile_counts_by_columns(e: np.ndarray, L: int, BM: int, BN: int):
    """The same counts as ``tile_counts`` without the L x L matrix: key j is
    visible to rows ``[j, min(e_j, L))``, so within a row block ``[i0, i1)`` it
    contributes ``max(0, min(i1, e_j, L) - max(i0, j))`` elements; the counts of
    a tile are those of its key columns summed.  Memory O(L) for long traces."""
    e = np.minimum(np.asarray(e, dtype=np.int64), L)
    nqt, nkt = -(-L // BM), -(-L // BN)
    j = np.arange(L)
    out = np.zeros((nqt, nkt), dtype=np.int64)
    pad = np.zeros(nkt * BN, dtype=np.int64)
    for qt in range(nqt):
        i0, i1 = qt * BM, min(qt * BM + BM, L)
        pad[:L] = np.maximum(np.minimum(i1, e) - np.maximum(i0, j), 0)
        out[qt] = pad.reshape(nkt, BN).sum(axis=1)
    return out


def class_totals(e: np.ndarray, lengths, BM: int, BN: int):
    """(EMPTY, FULL, PARTIAL) tile totals and the visible elements inside PARTIAL
    tiles, over packed traces, from ``tile_counts_by_columns``."""
    tot = np.zeros(3, dtype=np.int64)
    vis_partial, off = 0, 0
    for L in lengths:
        c = tile_counts_by_columns(e[off:off + L], L, BM, BN)
        full = c == BM * BN
        empty = c == 0
        tot += [int(empty.sum()), int(full.sum()), int((~full & ~empty).sum())]
        vis_partial += int(c[~full & ~empty].sum())
        off += L
    return tuple(int(x) for x in tot), vis_partial
