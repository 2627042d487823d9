"""Tile-class totals of the benchmark workloads at 128 x 128 tiles (and 64 x 64
for the 512-token trace), against counts tabulated independently of this code
before it was written, and the accounting that ties them to the visible-pair
count: BM * BN * #FULL + (visible elements of PARTIAL tiles) = visible pairs.

The counts come from ``oracle.tiles.tile_counts_by_columns``, which counts the
visible elements of every tile column by column from the mask definition
(key j is visible to rows [j, min(e_j, L)); Section 2, "KV-streams"); it is
pinned here to the per-element counter ``tile_counts`` on small traces.
"""
import numpy as np
import pytest

from oracle import attention as orc
from oracle import tiles as otiles
from paper_2609_35750_amd import inputs

# (EMPTY, FULL, PARTIAL) tiles per workload
TABLE = {
    ("trace512_tiny", 128): (6, 0, 10),
    ("trace512_tiny", 64): (38, 12, 14),
    ("trace16k_gqa4", 128): (12736, 3520, 128),
    ("trace32k_latest", 128): (59808, 5472, 256),
    ("varlen8_gqa5", 128): (91921, 14826, 1030),
    ("trace64k_last2", 128): (247524, 14108, 512),
}


def test_column_counter_equals_element_counter():
    rng = np.random.default_rng(11)
    for L in (1, 31, 64, 65, 200, 777):
        for e in (inputs.evict_at_random(L, rng), inputs.evict_at_layout(L, 5, 40, 9, "last2"),
                  np.full(L, L, dtype=np.int32)):
            for BM, BN in ((32, 64), (128, 128), (96, 64), (16, 128)):
                np.testing.assert_array_equal(otiles.tile_counts_by_columns(e, L, BM, BN),
                                              otiles.tile_counts(e, L, BM, BN))


@pytest.mark.parametrize("name,B", list(TABLE), ids=lambda x: str(x))
def test_tile_class_table(name, B):
    wl = inputs.WORKLOADS[name]
    e = wl.evict_at()
    (ne, nf, npart), vis_partial = otiles.class_totals(e, wl.lengths, B, B)
    assert (ne, nf, npart) == TABLE[(name, B)]
    # every visible pair lies in a FULL tile or is counted in a PARTIAL one
    off, pairs = 0, 0
    for L in wl.lengths:
        pairs += int((np.minimum(e[off:off + L].astype(np.int64), L) - np.arange(L)).sum())
        off += L
    assert B * B * nf + vis_partial == pairs
    if name == "trace512_tiny":
        assert pairs == orc.visible_pairs(e, wl.lengths) == 78080
