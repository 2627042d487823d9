"""Context-parallel shards through libkvs on the GPU (MI355X).

Each shard of query rows [r0, r1) runs the library's eviction-masked
forward and backward on its local trace [gathered keys; own tokens]
(paper_2609_35750_amd/shard.py); the owned rows' O, LSE, dQ are taken as is
and every local key's dK/dV is added into its owner's row (the backward's
reduce-scatter).  The assembled result must meet the parity bar against the
fp64 oracle of the whole trace: at small size element by element, at full
size (64k tokens, last-2 summaries, 8 shards at segment starts) at the
sampled positions of the committed checker fixture.
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import attention as orc
from paper_2609_35750_amd import inputs, shard
from tests.gpu_helpers import LSE_ABS, announce, assert_close, gpu_fwd_bwd, to_f64

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
           "dk": np.zeros((L, Hkv, D)), "dv": np.zeros((L, Hkv, D))}
    for p in plans:
        keys = torch.from_numpy(p.keys)
        ql = torch.cat([torch.zeros((p.n_g, Hq, D), dtype=q.dtype), q[p.r0:p.r1]])
        dol = torch.cat([torch.zeros((p.n_g, Hq, D), dtype=do.dtype), do[p.r0:p.r1]])
        r = gpu_fwd_bwd(kvs, ql, k[keys], v[keys], dol, p.evict_local, scale, B=1)
        out["O"][p.r0:p.r1] = to_f64(r["O"][p.n_g:])
        out["LSE"][:, p.r0:p.r1] = to_f64(r["LSE"][:, p.n_g:])
        out["dq"][p.r0:p.r1] = to_f64(r["dq"][p.n_g:])
        np.add.at(out["dk"], p.keys, to_f64(r["dk"]))
        np.add.at(out["dv"], p.keys, to_f64(r["dv"]))
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
    for key in ("O", "dq", "dk", "dv"):
        assert_close(f"cp {strategy}:{key}", got[key], ref[key])
    assert_close(f"cp {strategy}:LSE", got["LSE"], ref["LSE"], max_abs=LSE_ABS, rel_l2=1e-4, elementwise=False)


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
    G, rows, keys = wl.G, gold["rows"], gold["keys"]
    assert_close(f"cp {name}:O", got["O"][rows, :G], gold["O"])
    assert_close(f"cp {name}:dQ", got["dq"][rows, :G], gold["dQ"].astype(np.float64))
    assert_close(f"cp {name}:dK", got["dk"][keys, 0], gold["dK"])
    assert_close(f"cp {name}:dV", got["dv"][keys, 0], gold["dV"])
    assert_close(f"cp {name}:LSE", got["LSE"][:G][:, rows], gold["LSE"], max_abs=LSE_ABS, rel_l2=1e-4,
                 elementwise=False)
