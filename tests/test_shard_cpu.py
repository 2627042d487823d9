"""Context-parallel shards of one trace, CPU tier: the shard decomposition
(paper_2609_35750_amd/shard.py) run through the fp64 oracle shard by shard
reproduces the oracle on the whole trace, for every output.

A shard owns rows [r0, r1); it needs the earlier keys with e_j > r0 (still
live when its first token is generated).  Its local trace is [gathered keys;
own tokens] with e_local = e - r0 + n_g; the gathered rows carry dO = 0."""
import math

import numpy as np
import pytest
import torch

from oracle import attention as orc
from paper_2609_35750_amd import inputs, shard


def _run_shards(q, k, v, do, e, plans, scale):
    L, Hq, D = q.shape
    Hkv = k.shape[1]
    O = np.zeros((L, Hq, D))
    LSE = np.zeros((Hq, L))
    dq = np.zeros((L, Hq, D))
    dk = np.zeros((L, Hkv, D))
    dv = np.zeros((L, Hkv, D))
    for p in plans:
        keys = torch.from_numpy(p.keys)
        ql = torch.cat([torch.zeros((p.n_g, Hq, D), dtype=q.dtype), q[p.r0:p.r1]])
        dol = torch.cat([torch.zeros((p.n_g, Hq, D), dtype=do.dtype), do[p.r0:p.r1]])
        r = orc.backward(ql, k[keys], v[keys], p.evict_local, scale, dol)
        O[p.r0:p.r1] = r["O"][p.n_g:]
        LSE[:, p.r0:p.r1] = r["LSE"][:, p.n_g:]
        dq[p.r0:p.r1] = r["dq"][p.n_g:]
        np.add.at(dk, p.keys, r["dk"])          # the backward's reduce-scatter to the key owners
        np.add.at(dv, p.keys, r["dv"])
    return {"O": O, "LSE": LSE, "dq": dq, "dk": dk, "dv": dv}


@pytest.mark.parametrize("strategy", inputs.STRATEGIES)
@pytest.mark.parametrize("aligned", [True, False])
def test_shards_reproduce_the_whole_trace(strategy, aligned):
    L, p, w, s, Hq, Hkv, D = 260, 14, 40, 9, 4, 2, 16
    e = inputs.evict_at_layout(L, p, w, s, strategy)
    q, k, v, do = (inputs.randn_bf16(sh, 60 + i) for i, sh in
                   enumerate([(L, Hq, D), (L, Hkv, D), (L, Hkv, D), (L, Hq, D)]))
    scale = 1.0 / math.sqrt(D)
    cuts = inputs.segment_starts(L, p, w, s) if aligned else None
    plans = shard.plan_trace(e, 4, cuts)
    assert sum(pl.r1 - pl.r0 for pl in plans) == L
    got = _run_shards(q, k, v, do, e, plans, scale)
    ref = orc.backward(q, k, v, e, scale, do)
    for key in ("O", "LSE", "dq", "dk", "dv"):
        np.testing.assert_allclose(got[key], ref[key if key != "LSE" else "LSE"], rtol=1e-10, atol=1e-11)


def test_gathered_keys_are_the_live_retained_entries():
    """At segment-aligned cuts a shard gathers exactly the prompt and the
    summaries still live at its first row; evicted turns never travel."""
    L, p, w, s = 2000, 64, 200, 30
    for strategy, live_summaries in (("keep_all", None), ("latest_only", 1), ("last2", 2)):
        e = inputs.evict_at_layout(L, p, w, s, strategy)
        a = inputs.segment_starts(L, p, w, s)
        for pl in shard.plan_trace(e, 5, a):
            if pl.r0 == 0:
                assert pl.n_g == 0
                continue
            k = a.index(pl.r0)                  # the shard starts at segment k
            summaries = [np.arange(a[m] + w, a[m + 1]) for m in range(k)]
            if live_summaries is not None:
                summaries = summaries[-live_summaries:]
            expect = np.concatenate([np.arange(p)] + summaries)
            np.testing.assert_array_equal(pl.gathered, expect)
            # local indices are valid eviction indices: every key sees itself
            assert np.all(pl.evict_local > np.arange(pl.length))


def test_exchange_volume_counts():
    e = inputs.evict_at_layout(65536, 2048, 2048, 256, "last2")
    plans = shard.plan_trace(e, 8, inputs.segment_starts(65536, 2048, 2048, 256))
    vol = shard.exchange_volume(plans, 8, 128)
    assert vol["max_gathered_keys_per_shard"] == 2048 + 2 * 256
    assert vol["bytes_kv"] == vol["gathered_keys"] * 8 * 128 * 2 * 2


def test_row_work_counts_visible_pairs_and_balanced_cuts():
    e = inputs.evict_at_layout(3000, 100, 400, 60, "keep_all")
    work = shard.row_work(e)
    assert int(work.sum()) == orc.visible_pairs(e, [3000])
    cuts = inputs.segment_starts(3000, 100, 400, 60)
    plans = shard.plan_trace(e, 4, cuts, balance=True)
    assert [pl.r0 for pl in plans][1:] == sorted(set(pl.r0 for pl in plans[1:]))
    assert all(pl.r0 in cuts or pl.r0 == 0 for pl in plans)
    assert plans[-1].r1 == 3000 and sum(pl.r1 - pl.r0 for pl in plans) == 3000
