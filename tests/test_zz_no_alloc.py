"""The allocation-free forward (kvs_evict_attn_fwd_noalloc, called through the
C ABI) gives bit-identical O and LSE to the workspace-taking forward, on two
calls in a row (the second on a smaller, packed input, so the library scratch
holds the first call's statistics when it starts)."""
import ctypes

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


def _noalloc(kvs, q, k, v, ev, cu, B, ntok, max_seqlen, Hq, Hkv, D, scale):
    o = torch.empty_like(q)
    lse_shape = (B, Hq, max_seqlen) if cu is None else (Hq, ntok)
    lse = torch.empty(lse_shape, dtype=torch.float32, device=q.device)
    stream = torch.cuda.current_stream().cuda_stream
    st = kvs.lib.kvs_evict_attn_fwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), ev.data_ptr(),
                                            None if cu is None else cu.data_ptr(), o.data_ptr(), lse.data_ptr(),
                                            B, ntok, max_seqlen, Hq, Hkv, D, ctypes.c_float(scale), stream)
    assert st == kvs.KVS_OK, kvs.lib.kvs_last_error().decode()
    return o, lse


def _same(a, b):
    if a.dtype == torch.bfloat16:
        a, b = a.view(torch.int16), b.view(torch.int16)
    return torch.equal(a, b)


def test_noalloc_forward_matches_workspace_forward_twice(kvs):
    dev = torch.device("cuda:0")
    # call 1: two fixed-length traces of 2,000 tokens, D = 128, GQA 4
    wl = inputs.custom_workload("noalloc_a", 8, 2, 128, [2000, 2000], 64, 400, 50, "last2", varlen=False, seed=71)
    announce(f"noalloc call 1: {wl.lengths} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D}")
    t = inputs.make_tensors(wl, with_grad=False)
    B, T = wl.B, wl.T
    q, k, v = (t[x].to(dev).view(B, T, -1, wl.D) for x in ("q", "k", "v"))
    ev = torch.from_numpy(wl.evict_at()).to(dev).view(B, T)
    o_ref, lse_ref = kvs.kvs_evict_attn_fwd(q, k, v, ev, wl.softmax_scale)
    o, lse = _noalloc(kvs, q, k, v, ev, None, B, B * T, T, wl.Hq, wl.Hkv, wl.D, wl.softmax_scale)
    torch.cuda.synchronize()
    assert _same(o, o_ref) and _same(lse, lse_ref)
    # call 2: smaller, packed (ragged tails, a 1-token trace), D = 64, no prompt
    wl2 = inputs.custom_workload("noalloc_b", 6, 3, 64, [300, 1, 129], 0, 40, 8, "keep_all", varlen=True, seed=72)
    announce(f"noalloc call 2: {wl2.lengths} Hq={wl2.Hq} Hkv={wl2.Hkv} D={wl2.D}")
    t2 = inputs.make_tensors(wl2, with_grad=False)
    q2, k2, v2 = (t2[x].to(dev) for x in ("q", "k", "v"))
    ev2 = torch.from_numpy(wl2.evict_at()).to(dev)
    cu2 = torch.from_numpy(wl2.cu_seqlens()).to(dev)
    o2, lse2 = _noalloc(kvs, q2, k2, v2, ev2, cu2, wl2.B, wl2.ntok, wl2.T, wl2.Hq, wl2.Hkv, wl2.D,
                        wl2.softmax_scale)
    o2_ref, lse2_ref = kvs.kvs_evict_attn_fwd(q2, k2, v2, ev2, wl2.softmax_scale, cu2, wl2.T)
    torch.cuda.synchronize()
    assert _same(o2, o2_ref) and _same(lse2, lse2_ref)
    assert torch.isfinite(o2.float()).all() and torch.isfinite(lse2).all()
    print("[no-alloc] two calls bit-identical to the workspace forward", flush=True)
