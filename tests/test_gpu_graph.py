"""Forward + backward captured in a HIP graph (the benchmark's --graph mode):
every replay, with other eager work and synchronisations between replays,
gives outputs bit-identical to the eager calls on the same inputs."""
import numpy as np
import pytest
import torch

from paper_2609_35750_amd import inputs
from tests.gpu_helpers import announce

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kvs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35750_amd import kvs as k

    return k


@pytest.mark.parametrize("varlen", [False, True])
def test_graph_replays_match_eager(kvs, varlen):
    dev = torch.device("cuda:0")
    lengths = [9000] if not varlen else [700, 8500, 129]   # split key blocks included
    wl = inputs.custom_workload("graph", 8, 2, 128, lengths, 256, 1500, 100, "last2", varlen=varlen, seed=91)
    announce(f"graph replay lengths={lengths}")
    t = inputs.make_tensors(wl)
    e = wl.evict_at()
    if varlen:
        q, k, v, do = (t[x].to(dev) for x in ("q", "k", "v", "do"))
        ev = torch.from_numpy(e).to(dev)
        cu = torch.from_numpy(wl.cu_seqlens()).to(dev)
        kvs.kvs_evict_attn_fwd(q, k, v, ev, wl.softmax_scale, cu, wl.T)   # host check of cu_seqlens, once
        # no host copy of cu_seqlens inside the capture (a device-to-host copy cannot be captured)
        kw = dict(cu_seqlens=cu, max_seqlen=wl.T, check_cu=False)
    else:
        shp = lambda x: x.to(dev).view(1, wl.T, x.shape[1], wl.D)
        q, k, v, do = (shp(t[x]) for x in ("q", "k", "v", "do"))
        ev = torch.from_numpy(e).to(dev).view(1, wl.T)
        kw = {}
    outs = [torch.empty_like(q), torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)]
    state = {}

    def step():
        o, lse = kvs.kvs_evict_attn_fwd(q, k, v, ev, wl.softmax_scale, out=outs[0], **kw)
        kvs.kvs_evict_attn_bwd(do, q, k, v, o, lse, ev, wl.softmax_scale, dq=outs[1], dk=outs[2], dv=outs[3], **kw)
        state["lse"] = lse

    step()
    torch.cuda.synchronize()
    ref = [x.clone() for x in outs] + [state["lse"].clone()]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(4):
        for x in outs:
            x.fill_(float("nan"))          # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = outs + [state["lse"]]
        for name, a, b in zip(("O", "dQ", "dK", "dV", "LSE"), got, ref):
            av = a.view(torch.int16) if a.dtype == torch.bfloat16 else a
            bv = b.view(torch.int16) if b.dtype == torch.bfloat16 else b
            assert torch.equal(av, bv), f"replay {r}: {name} differs from the eager call"
    print(f"[graph] {lengths}: 4 replays bit-identical to the eager calls", flush=True)
