"""Context-parallel shards through libkvs on the GPU (MI355X).

Each shard of query rows [r0, r1) runs the library's eviction-masked
forward and backward on its local trace [gathered keys; own tokens]
(paper_2609_35750_amd/shard.py); the owned rows' O, LSE, dQ are taken as is
and every local key's dK/dV is added into its owner's row (the backward's
reduce-scatter).  The assembled result must meet the parity bar against the
fp64 oracle of the whole trace: at small size element by element, at full
size (64k tokens, last-2 summaries, 8 shards at segment starts) at the
sampled positions of the committed oracle fixture.
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import attention as orc
from paper_2609_35750_amd import inputs, shard
from tests.gpu_helpers import announce, assert_close, assert_lse, gpu_fwd_bwd, to_f64, ulp_bf16

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def kvs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35750_amd import kvs as k

    return k


def _assemble(kvs, q, k, v, do, plans, scale):
    L, Hq, D = q.shape
    Hkv = k.shape[1]
    out = {"O": np.zeros((L, Hq, D)), "LSE": np.zeros((Hq, L)), "dq": np.zeros((L, Hq, D)),
           "dk": np.zeros((L, Hkv, D)), "dv": np.zeros((L, Hkv, D)),
           # half a bf16 spacing per shard partial added into a key (the partials are bf16 outputs;
           # a reduce-scatter would add fp32 partials instead)
           "round_dk": np.zeros((L, Hkv, D)), "round_dv": np.zeros((L, Hkv, D))}
    for p in plans:
        keys = torch.from_numpy(p.keys)
        ql = torch.cat([torch.zeros((p.n_g, Hq, D), dtype=q.dtype), q[p.r0:p.r1]])
        dol = torch.cat([torch.zeros((p.n_g, Hq, D), dtype=do.dtype), do[p.r0:p.r1]])
        r = gpu_fwd_bwd(kvs, ql, k[keys], v[keys], dol, p.evict_local, scale, B=1)
        out["O"][p.r0:p.r1] = to_f64(r["O"][p.n_g:])
        out["LSE"][:, p.r0:p.r1] = to_f64(r["LSE"][:, p.n_g:])
        out["dq"][p.r0:p.r1] = to_f64(r["dq"][p.n_g:])
        dk_s, dv_s = to_f64(r["dk"]), to_f64(r["dv"])
        np.add.at(out["dk"], p.keys, dk_s)
        np.add.at(out["dv"], p.keys, dv_s)
        np.add.at(out["round_dk"], p.keys, 0.5 * ulp_bf16(dk_s))
        np.add.at(out["round_dv"], p.keys, 0.5 * ulp_bf16(dv_s))
    return out


@pytest.mark.parametrize("strategy,aligned,n", [("last2", True, 4), ("keep_all", False, 3), ("latest_only", True, 5)])
def test_shards_match_the_whole_trace(kvs, strategy, aligned, n):
    L, p, w, s, Hq, Hkv, D = 3000, 100, 400, 60, 8, 2, 128
    announce(f"cp shards L={L} {strategy} aligned={aligned} n={n} Hq={Hq} Hkv={Hkv} D={D}")
    e = inputs.evict_at_layout(L, p, w, s, strategy)
    q, k, v, do = (inputs.randn_bf16(sh, 500 + i) for i, sh in
                   enumerate([(L, Hq, D), (L, Hkv, D), (L, Hkv, D), (L, Hq, D)]))
    scale = 1.0 / math.sqrt(D)
    plans = shard.plan_trace(e, n, inputs.segment_starts(L, p, w, s) if aligned else None)
    got = _assemble(kvs, q, k, v, do, plans, scale)
    ref = orc.backward(q, k, v, e, scale, do)
    E = orc.dq_rounding_scale(q, k, v, e, scale, do, np.arange(L))
    assert_close(f"cp {strategy}:O", got["O"], ref["O"])
    assert_close(f"cp {strategy}:dq", got["dq"], ref["dq"], E=E)
    assert_close(f"cp {strategy}:dk", got["dk"], ref["dk"], extra=got["round_dk"])
    assert_close(f"cp {strategy}:dv", got["dv"], ref["dv"], extra=got["round_dv"])
    assert_lse(f"cp {strategy}", got["LSE"], ref["LSE"])


def test_fullsize_64k_eight_shards_sampled(kvs):
    name = "trace64k_last2"
    path = os.path.join(GOLDEN, f"parity_{name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"{path} not generated")
    gold = np.load(path)
    wl = inputs.WORKLOADS[name]
    e = wl.evict_at()
    plans = shard.plan_trace(e, 8, inputs.segment_starts(wl.T, wl.p, wl.w, wl.s))
    announce(f"cp full-size {name}: 8 shards, gathered keys per shard {[pl.n_g for pl in plans]}")
    t = inputs.make_tensors(wl)
    got = _assemble(kvs, t["q"], t["k"], t["v"], t["do"], plans, wl.softmax_scale)
    G, rows, keys, kvh = wl.G, gold["rows"], gold["keys"], gold["kv_heads"]
    heads = np.concatenate([np.arange(g * G, (g + 1) * G) for g in kvh])
    assert_close(f"cp {name}:O", got["O"][rows][:, heads], gold["O"])
    assert_close(f"cp {name}:dQ", got["dq"][rows][:, heads], gold["dQ"], E=gold["E_dQ"])
    assert_close(f"cp {name}:dK", got["dk"][keys][:, kvh], gold["dK"], extra=got["round_dk"][keys][:, kvh])
    assert_close(f"cp {name}:dV", got["dv"][keys][:, kvh], gold["dV"], extra=got["round_dv"][keys][:, kvh])
    assert_lse(f"cp {name}", got["LSE"][heads][:, rows], gold["LSE"])
