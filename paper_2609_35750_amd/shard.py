"""Context-parallel shards of one continuous trace (host-side index bookkeeping).

One long trace can be split across GPUs by its query rows.  Shard r owns the
rows ``[r0, r1)`` and their keys; because query ``i`` sees key ``j`` iff
``j <= i < e_j``, a key ``j < r0`` of an earlier shard is needed by shard r
iff ``e_j > r0`` (it is still live when the shard's first token is
generated): the retained prompt and summaries, and the turns of a segment
the cut falls into.  Evicted keys never travel (Section 2, "KV-streams": the
engine drops them for good).  Cutting at segment boundaries keeps that set
to the prompt plus the live summaries.

On one GPU a shard is the eviction-masked attention of a local trace
``[gathered keys ; own tokens]`` with the eviction indices moved into local
coordinates, ``e_local = e - r0 + n_g`` (clipped to the local length).  The
gathered keys' own rows are padding: their dO is zero, so they add nothing
to any gradient and their outputs are dropped.  Summing every shard's dK/dV
rows into the owning key's row is the reduce-scatter of the backward.

This module holds only index arithmetic; the attention itself runs in libkvs.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np


@dataclasses.dataclass
class ShardPlan:
    r0: int                  # first owned row (trace position)
    r1: int                  # one past the last owned row
    gathered: np.ndarray     # positions of the earlier keys the shard needs (increasing)
    evict_local: np.ndarray  # int32 [n_g + r1 - r0]: eviction index of each local key, local coordinates

    @property
    def n_g(self) -> int:
        return int(self.gathered.size)

    @property
    def keys(self) -> np.ndarray:
        """Trace position of every local key: the gathered keys, then the owned rows."""
        return np.concatenate([self.gathered, np.arange(self.r0, self.r1, dtype=np.int64)])

    @property
    def length(self) -> int:
        return self.n_g + self.r1 - self.r0


def shard_rows(L: int, n_shards: int, cuts: Optional[Sequence[int]] = None) -> List[Tuple[int, int]]:
    """``n_shards`` contiguous row ranges covering ``[0, L)``: equal splits, each
    interior cut moved to the nearest candidate in ``cuts`` (e.g. segment starts)
    when one is given; empty ranges are dropped."""
    if n_shards < 1:
        raise ValueError("n_shards must be >= 1")
    bounds = [0]
    cand = np.asarray(sorted(set(int(c) for c in cuts if 0 < c < L)), dtype=np.int64) if cuts is not None else None
    for r in range(1, n_shards):
        x = (L * r) // n_shards
        if cand is not None and cand.size:
            x = int(cand[np.argmin(np.abs(cand - x))])
        bounds.append(max(x, bounds[-1]))
    bounds.append(L)
    return [(a, b) for a, b in zip(bounds[:-1], bounds[1:]) if b > a]


def shard_plan(evict_at, r0: int, r1: int) -> ShardPlan:
    """Keys shard ``[r0, r1)`` of a trace needs, and their local eviction indices."""
    e = np.asarray(evict_at, dtype=np.int64)
    L = e.size
    if not 0 <= r0 < r1 <= L:
        raise ValueError("need 0 <= r0 < r1 <= L")
    gathered = np.nonzero(e[:r0] > r0)[0].astype(np.int64)
    keys = np.concatenate([gathered, np.arange(r0, r1, dtype=np.int64)])
    n_g = gathered.size
    n_loc = n_g + r1 - r0
    local = np.minimum(e[keys], r1) - r0 + n_g          # e_j >= r1 means "never" inside the shard
    local = np.minimum(local, n_loc)
    return ShardPlan(r0, r1, gathered, local.astype(np.int32))


def row_work(evict_at) -> np.ndarray:
    """Keys each query row sees (key j counts on rows j .. e_j - 1)."""
    e = np.minimum(np.asarray(evict_at, dtype=np.int64), len(evict_at))
    L = e.size
    diff = np.zeros(L + 1, dtype=np.int64)
    np.add.at(diff, np.arange(L), 1)
    np.add.at(diff, e, -1)
    return np.cumsum(diff[:L])


def balanced_rows(evict_at, n_shards: int, cuts: Sequence[int]) -> List[Tuple[int, int]]:
    """Row ranges with about equal attention work (visible pairs): cut r goes to
    the candidate in ``cuts`` whose cumulative work is closest to r / n_shards of
    the total; empty ranges are dropped."""
    work = np.concatenate([[0], np.cumsum(row_work(evict_at))])
    L = len(evict_at)
    cand = np.asarray(sorted(set(int(c) for c in cuts if 0 < c < L)), dtype=np.int64)
    bounds = [0]
    for r in range(1, n_shards):
        target = work[-1] * r / n_shards
        x = int(cand[np.argmin(np.abs(work[cand] - target))]) if cand.size else (L * r) // n_shards
        bounds.append(max(x, bounds[-1]))
    bounds.append(L)
    return [(a, b) for a, b in zip(bounds[:-1], bounds[1:]) if b > a]


def plan_trace(evict_at, n_shards: int, cuts: Optional[Sequence[int]] = None, balance: bool = False) -> List[ShardPlan]:
    """Shard plans of a trace: equal row ranges, or ranges of equal work
    (``balance``), with cuts at candidate positions (segment starts) if given."""
    e = np.asarray(evict_at)
    if balance:
        rows = balanced_rows(e, n_shards, cuts if cuts is not None else range(1, e.size))
    else:
        rows = shard_rows(e.size, n_shards, cuts)
    return [shard_plan(e, a, b) for a, b in rows]


def exchange_volume(plans: Sequence[ShardPlan], Hkv: int, D: int, bytes_per_elem: int = 2) -> dict:
    """Keys moved by the forward all-gather (and back by the backward's
    reduce-scatter of their dK/dV), in keys and bytes (K and V)."""
    keys = int(sum(p.n_g for p in plans))
    return {"gathered_keys": keys, "max_gathered_keys_per_shard": int(max(p.n_g for p in plans)),
            "bytes_kv": keys * Hkv * D * bytes_per_elem * 2}
