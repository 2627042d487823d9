"""The autograd wrapper (``kvs.evict_attn``) on the GPU (MI355X).

Gradients through ``torch.autograd`` must be exactly those of the explicit
forward and backward calls (same kernels, same inputs), and match the fp64
oracle; LSE is returned without a gradient.  Every case prints its name
before it runs.
"""
import numpy as np
import pytest
import torch

from oracle import attention as orc
from paper_2609_35750_amd import inputs
from tests.gpu_helpers import assert_close, announce, to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kvs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35750_amd import kvs as k

    return k


@pytest.mark.parametrize("varlen", [False, True], ids=["fixed", "varlen"])
def test_autograd_matches_explicit_calls_and_oracle(kvs, varlen):
    lengths = [300, 300] if not varlen else [257, 1, 130]
    wl = inputs.custom_workload("autograd", 8, 2, 128, lengths, 12, 60, 10, "last2", varlen=varlen, seed=61)
    announce(f"autograd {wl.name} lengths={lengths} varlen={varlen}")
    dev = torch.device("cuda:0")
    t = inputs.make_tensors(wl)
    e = wl.evict_at()
    n, B, T = wl.ntok, len(lengths), lengths[0]
    shp = (lambda x: x.view(B, T, x.shape[1], x.shape[2])) if not varlen else (lambda x: x)
    q, k, v, do = (shp(t[x].to(dev)) for x in ("q", "k", "v", "do"))
    ev = torch.from_numpy(e).to(dev)
    ev = ev.view(B, T) if not varlen else ev
    cu = torch.from_numpy(wl.cu_seqlens()).to(dev) if varlen else None
    mx = max(lengths) if varlen else None

    qg, kg, vg = (x.clone().requires_grad_(True) for x in (q, k, v))
    o, lse = kvs.evict_attn(qg, kg, vg, ev, wl.softmax_scale, cu, mx)
    assert not lse.requires_grad
    o.backward(do)

    o2, lse2 = kvs.kvs_evict_attn_fwd(q, k, v, ev, wl.softmax_scale, cu, mx)
    dq2, dk2, dv2 = kvs.kvs_evict_attn_bwd(do, q, k, v, o2, lse2, ev, wl.softmax_scale, cu, mx)
    torch.cuda.synchronize()
    assert torch.equal(o.detach(), o2) and torch.equal(lse, lse2)
    for name, g, ref in (("dQ", qg.grad, dq2), ("dK", kg.grad, dk2), ("dV", vg.grad, dv2)):
        assert torch.equal(g, ref), f"{name}: autograd differs from the explicit backward"

    ref = orc.backward(t["q"], t["k"], t["v"], e, wl.softmax_scale, t["do"],
                       cu_seqlens=wl.cu_seqlens() if varlen else np.arange(B + 1) * T)
    flat = lambda x: to_f64(x.reshape(n, x.shape[-2], x.shape[-1]))
    assert_close("autograd O", flat(o.detach()), ref["O"])
    E = orc.dq_rounding_scale(t["q"], t["k"], t["v"], e, wl.softmax_scale, t["do"], np.arange(n),
                              cu_seqlens=wl.cu_seqlens() if varlen else np.arange(B + 1) * T)
    assert_close("autograd dQ", flat(qg.grad), ref["dq"], E=E)
    assert_close("autograd dK", flat(kg.grad), ref["dk"])
    assert_close("autograd dV", flat(vg.grad), ref["dv"])
