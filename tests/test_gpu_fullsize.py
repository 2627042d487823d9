"""Full-size workloads: the HIP path at the exact launch configuration the
benchmark times, compared with the fp64 oracle at sampled positions, and the
tile-classifier shortcuts checked bit for bit over the whole tensors.

The expected values come from ``tests/golden/make_parity_fixtures.py`` (which
runs only the oracle, for the q-heads of the first and the last KV head).
Bound (tests/gpu_helpers.py): |x - x*| <= 2e-2 + 0.45 ulp_bf16(x*) per
element (+ 2^-8 E for dQ, E the oracle's first-order sensitivity of dQ to
the bf16 roundings of O and dS) and relative L2 <= 1e-2 for O, dQ, dK, dV;
LSE within 1e-3 absolute.  Every comparison prints its flat max |x - x*|
against 2e-2, its worst error / bound and its relative L2.

The mask must block every deleted span (Section 2, "KV-streams"): a skipped
EMPTY tile must hold no visible entry and an unmasked FULL tile no masked one.
One leaked key moves an output by far less than any tolerance, so the
shortcuts are checked exactly: the same calls with every EMPTY tile processed
(masked) and with every FULL tile masked must give bit-identical O, LSE, dQ,
dK and dV over the whole tensors.
"""
import dataclasses
import os

import numpy as np
import pytest
import torch

from oracle import attention as orc
from paper_2609_35750_amd import inputs
from tests.gpu_helpers import REL_L2, announce, assert_close, assert_lse, to_f64

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
NAMES = ["trace16k_gqa4", "trace32k_latest", "varlen8_gqa5", "trace64k_last2", "textworld32k_sliding"]
BITWISE = ["trace16k_gqa4", "trace32k_latest", "varlen8_gqa5", "trace64k_last2"]


@pytest.fixture(scope="module")
def kvs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35750_amd import kvs as k

    return k


def _device_inputs(wl):
    dev = torch.device("cuda:0")
    t = inputs.make_tensors(wl)
    e = wl.evict_at()
    if wl.varlen:
        q, k, v, do = (t[x].to(dev) for x in ("q", "k", "v", "do"))
        ev = torch.from_numpy(e).to(dev)
        kw = dict(cu_seqlens=torch.from_numpy(wl.cu_seqlens()).to(dev), max_seqlen=wl.T)
    else:
        shp = lambda x: x.to(dev).view(1, wl.T, x.shape[1], wl.D)
        q, k, v, do = (shp(t[x]) for x in ("q", "k", "v", "do"))
        ev = torch.from_numpy(e).to(dev).view(1, wl.T)
        kw = {}
    return (q, k, v, do, ev, kw)


def _run(kvs, wl, dev_in, flags=0):
    q, k, v, do, ev, kw = dev_in
    o, lse = kvs.kvs_evict_attn_fwd(q, k, v, ev, wl.softmax_scale, flags=flags, **kw)
    dq, dk, dv = kvs.kvs_evict_attn_bwd(do, q, k, v, o, lse, ev, wl.softmax_scale, flags=flags, **kw)
    torch.cuda.synchronize()
    flat = lambda x: x.reshape(wl.ntok, x.shape[-2], x.shape[-1])
    lse_p = lse if wl.varlen else lse.permute(1, 0, 2).reshape(wl.Hq, wl.ntok)
    return {"O": flat(o), "LSE": lse_p, "dq": flat(dq), "dk": flat(dk), "dv": flat(dv)}


@pytest.mark.parametrize("name", NAMES)
def test_fullsize_sampled_parity(kvs, name):
    path = os.path.join(GOLDEN, f"parity_{name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"{path} not generated")
    gold = np.load(path)
    wl = inputs.WORKLOADS[name]
    announce(f"full-size {name}: tokens={wl.ntok} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D}")
    res = _run(kvs, wl, _device_inputs(wl))
    for key in ("O", "LSE", "dq", "dk", "dv"):
        assert torch.isfinite(res[key].float()).all(), f"{name}: non-finite {key}"
    G = wl.G
    rows, keys = gold["rows"], gold["keys"]
    heads = np.concatenate([np.arange(g * G, (g + 1) * G) for g in gold["kv_heads"]])
    rows_t, keys_t = torch.from_numpy(rows).cuda(), torch.from_numpy(keys).cuda()
    heads_t, kvh_t = torch.from_numpy(heads).cuda(), torch.from_numpy(gold["kv_heads"]).cuda()
    pick = lambda x, r, h: to_f64(x.index_select(0, r).index_select(1, h))
    assert_close(f"{name}:O", pick(res["O"], rows_t, heads_t), gold["O"])
    assert_close(f"{name}:dQ", pick(res["dq"], rows_t, heads_t), gold["dQ"], E=gold["E_dQ"])
    assert_close(f"{name}:dK", pick(res["dk"], keys_t, kvh_t), gold["dK"])
    assert_close(f"{name}:dV", pick(res["dv"], keys_t, kvh_t), gold["dV"])
    assert_lse(name, to_f64(res["LSE"].index_select(0, heads_t).index_select(1, rows_t)), gold["LSE"])
    # whole-tensor norms of each checked KV head's outputs (every row, every key) against the oracle's
    for i, g in enumerate(gold["kv_heads"]):
        hs = slice(g * G, (g + 1) * G)
        for key, gkey, sl in (("O", "norm_O", hs), ("dq", "norm_dQ", hs), ("dk", "norm_dK", slice(g, g + 1)),
                              ("dv", "norm_dV", slice(g, g + 1))):
            n = float(torch.linalg.vector_norm(res[key][:, sl].double()))
            want = float(gold[gkey][i])
            assert abs(n - want) <= REL_L2 * want, (name, key, g, n, want)


@pytest.mark.parametrize("name", BITWISE)
def test_fullsize_tile_shortcuts_are_exact(kvs, name):
    wl = inputs.WORKLOADS[name]
    announce(f"full-size switches {name}: tokens={wl.ntok}")
    dev_in = _device_inputs(wl)
    base = _run(kvs, wl, dev_in)
    for flags in (kvs.FLAG_NO_EMPTY_SKIP, kvs.FLAG_FULL_AS_PARTIAL):
        other = _run(kvs, wl, dev_in, flags=flags)
        for key in ("O", "LSE", "dq", "dk", "dv"):
            a, b = base[key], other[key]
            if a.dtype == torch.bfloat16:
                a, b = a.view(torch.int16), b.view(torch.int16)
            assert torch.equal(a, b), f"{name}: {key} differs bitwise with flags {flags}"
        del other
        print(f"[bitwise] {name}: flags {flags}: O, LSE, dQ, dK, dV identical over the whole tensors", flush=True)


def _fewest_rows_keys(keys, e, cu, ntok, count=8):
    """The ``count`` sampled keys seen by the fewest rows (their sums stay cheap for every head)."""
    span = np.empty(keys.size, dtype=np.int64)
    for c, j in enumerate(keys):
        b = int(np.searchsorted(cu, j, side="right")) - 1 if cu is not None else 0
        start = int(cu[b]) if cu is not None else 0
        L = int(cu[b + 1] - cu[b]) if cu is not None else ntok
        span[c] = min(int(e[j]), L) - (int(j) - start)
    return np.sort(keys[np.argsort(span, kind="stable")[:count]])


@pytest.mark.parametrize("name", NAMES)
def test_fullsize_every_head_sampled(kvs, name):
    """Every q-head and every KV head at the benchmarked launch configuration:
    O, LSE and dQ at the fixture's sampled rows for all q-heads, and dK, dV for
    all KV heads at the sampled keys seen by the fewest rows, against the
    oracle's row- and key-sampled forms evaluated here."""
    path = os.path.join(GOLDEN, f"parity_{name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"{path} not generated")
    gold = np.load(path)
    wl = inputs.WORKLOADS[name]
    announce(f"full-size every head {name}: tokens={wl.ntok} Hq={wl.Hq} Hkv={wl.Hkv}")
    t = inputs.make_tensors(wl)
    e = wl.evict_at()
    cu = wl.cu_seqlens() if wl.varlen else None
    res = _run(kvs, wl, _device_inputs(wl))
    rows = gold["rows"]
    ref = orc.rows_reference(t["q"], t["k"], t["v"], e, wl.softmax_scale, t["do"], rows, cu_seqlens=cu)
    rows_t = torch.from_numpy(rows).cuda()
    assert_close(f"{name}:O all heads", to_f64(res["O"].index_select(0, rows_t)), ref["O"])
    assert_close(f"{name}:dQ all heads", to_f64(res["dq"].index_select(0, rows_t)), ref["dq"], E=ref["E"])
    assert_lse(f"{name} all heads", to_f64(res["LSE"].index_select(1, rows_t)), ref["LSE"])
    pick = _fewest_rows_keys(gold["keys"], e, cu, wl.ntok)
    dk_ref, dv_ref = orc.keys_reference(t["q"], t["k"], t["v"], e, wl.softmax_scale, t["do"], pick, cu_seqlens=cu)
    keys_t = torch.from_numpy(pick).cuda()
    assert_close(f"{name}:dK all KV heads", to_f64(res["dk"].index_select(0, keys_t)), dk_ref)
    assert_close(f"{name}:dV all KV heads", to_f64(res["dv"].index_select(0, keys_t)), dv_ref)


@pytest.mark.parametrize("name", ["trace16k_gqa4", "varlen8_gqa5"])
def test_fullsize_head_dim_64(kvs, name):
    """The D = 64 kernels at full size (same layouts, head dimension 64): every
    q-head at the fixture's sampled rows, every KV head at the sampled keys
    seen by the fewest rows, against the sampled oracle; finiteness and the
    tile-classifier switches bit for bit over the whole tensors."""
    gold = np.load(os.path.join(GOLDEN, f"parity_{name}.npz"))
    wl = dataclasses.replace(inputs.WORKLOADS[name], D=64)
    announce(f"full-size D=64 {name}: tokens={wl.ntok} Hq={wl.Hq} Hkv={wl.Hkv}")
    t = inputs.make_tensors(wl)
    e = wl.evict_at()
    cu = wl.cu_seqlens() if wl.varlen else None
    dev_in = _device_inputs(wl)
    res = _run(kvs, wl, dev_in)
    for key in ("O", "LSE", "dq", "dk", "dv"):
        assert torch.isfinite(res[key].float()).all(), f"{name} D=64: non-finite {key}"
    for flags in (kvs.FLAG_NO_EMPTY_SKIP, kvs.FLAG_FULL_AS_PARTIAL):
        other = _run(kvs, wl, dev_in, flags=flags)
        for key in ("O", "LSE", "dq", "dk", "dv"):
            a, b = res[key], other[key]
            if a.dtype == torch.bfloat16:
                a, b = a.view(torch.int16), b.view(torch.int16)
            assert torch.equal(a, b), f"{name} D=64: {key} differs bitwise with flags {flags}"
        del other
    rows = gold["rows"]
    ref = orc.rows_reference(t["q"], t["k"], t["v"], e, wl.softmax_scale, t["do"], rows, cu_seqlens=cu)
    rows_t = torch.from_numpy(rows).cuda()
    assert_close(f"{name} D=64:O", to_f64(res["O"].index_select(0, rows_t)), ref["O"])
    assert_close(f"{name} D=64:dQ", to_f64(res["dq"].index_select(0, rows_t)), ref["dq"], E=ref["E"])
    assert_lse(f"{name} D=64", to_f64(res["LSE"].index_select(1, rows_t)), ref["LSE"])
    pick = _fewest_rows_keys(gold["keys"], e, cu, wl.ntok)
    dk_ref, dv_ref = orc.keys_reference(t["q"], t["k"], t["v"], e, wl.softmax_scale, t["do"], pick, cu_seqlens=cu)
    keys_t = torch.from_numpy(pick).cuda()
    assert_close(f"{name} D=64:dK", to_f64(res["dk"].index_select(0, keys_t)), dk_ref)
    assert_close(f"{name} D=64:dV", to_f64(res["dv"].index_select(0, keys_t)), dv_ref)
