"""The pins are discriminating: planting a plausible mistake in a copy of the
CPU oracle (a dropped term, a wrong sign, index or boundary, a missing scale)
makes at least one pin fail.  CPU only; the oracle itself is untouched."""
import math
import os
import types

import numpy as np
import pytest
import torch

from oracle import stream_sim
from paper_2609_35750_amd import inputs

SRC = open(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "attention.py")).read()

MUTATIONS = {
    "mask boundary i <= e_j": ("(j <= i) & (i < ej)", "(j <= i) & (i <= ej)"),
    "diagonal excluded": ("(j <= i) & (i < ej)", "(j < i) & (i < ej)"),
    "GQA map h % Hkv": ("        g = h // G\n        for i0 in range(0, L, ROW_BLOCK):\n            i1 = min(i0 + ROW_BLOCK, L)\n            M = visible_mask(e, L, i0, i1, i1)\n            S = scale * (q[i0:i1, h, :] @ k[:i1, g, :].T)\n            S = np.where(M, S, -np.inf)\n            m = S.max(axis=1, keepdims=True)\n            E = np.where(M, np.exp(S - m), 0.0)\n            l = E.sum(axis=1, keepdims=True)\n            P = E / l\n            O[i0:i1, h, :] = P @ v[:i1, g, :]\n            LSE[h, i0:i1] = (m + np.log(l))[:, 0]\n            dP",
                        "        g = h % Hkv\n        for i0 in range(0, L, ROW_BLOCK):\n            i1 = min(i0 + ROW_BLOCK, L)\n            M = visible_mask(e, L, i0, i1, i1)\n            S = scale * (q[i0:i1, h, :] @ k[:i1, g, :].T)\n            S = np.where(M, S, -np.inf)\n            m = S.max(axis=1, keepdims=True)\n            E = np.where(M, np.exp(S - m), 0.0)\n            l = E.sum(axis=1, keepdims=True)\n            P = E / l\n            O[i0:i1, h, :] = P @ v[:i1, g, :]\n            LSE[h, i0:i1] = (m + np.log(l))[:, 0]\n            dP"),
    "dK without scale": ("dk[:i1, g, :] += scale * (dS.T @ q[i0:i1, h, :])", "dk[:i1, g, :] += dS.T @ q[i0:i1, h, :]"),
    "dQ without scale": ("dq[i0:i1, h, :] = scale * (dS @ k[:i1, g, :])", "dq[i0:i1, h, :] = dS @ k[:i1, g, :]"),
    "Delta dropped": ("dS = P * (dP - dlt)", "dS = P * dP"),
    "dS sign": ("dS = P * (dP - dlt)", "dS = P * (dlt - dP)"),
    "dV from dS": ("dv[:i1, g, :] += P.T @ do[i0:i1, h, :]", "dv[:i1, g, :] += dS.T @ do[i0:i1, h, :]"),
    "dQ overwrites across heads": ("dq[i0:i1, h, :] = scale", "dq[i0:i1, 0, :] = scale"),
    "LSE without log": ("LSE[h, i0:i1] = (m + np.log(l))[:, 0]\n            dP", "LSE[h, i0:i1] = (m + l)[:, 0]\n            dP"),
    "LSE without max": ("LSE[h, i0:i1] = (m + np.log(l))[:, 0]\n            dP", "LSE[h, i0:i1] = np.log(l)[:, 0]\n            dP"),
    "forward unscaled": ("            S = scale * (q[i0:i1, h, :] @ k[:i1, g, :].T)\n            S = np.where(M, S, -np.inf)\n            m = S.max(axis=1, keepdims=True)\n            E = np.where(M, np.exp(S - m), 0.0)\n            l = E.sum(axis=1, keepdims=True)\n            P = E / l\n            O[i0:i1, h, :] = P @ v[:i1, g, :]\n            LSE[h, i0:i1] = (m + np.log(l))[:, 0]\n    return O, LSE",
                         "            S = q[i0:i1, h, :] @ k[:i1, g, :].T\n            S = np.where(M, S, -np.inf)\n            m = S.max(axis=1, keepdims=True)\n            E = np.where(M, np.exp(S - m), 0.0)\n            l = E.sum(axis=1, keepdims=True)\n            P = E / l\n            O[i0:i1, h, :] = P @ v[:i1, g, :]\n            LSE[h, i0:i1] = (m + np.log(l))[:, 0]\n    return O, LSE"),
    "eviction index ignored": ("ej = np.minimum(e[:j1].astype(np.int64), L)[None, :]", "ej = np.full((1, j1), L)"),
    "sampled rows: diagonal excluded": ("np.minimum(e_tr[:i + 1], L) > i", "np.minimum(e_tr[:i], L) > i"),
    "sampled keys: rows past the eviction": ("(il[:, None] < et[cand][None, :])", "(il[:, None] <= et[cand][None, :])"),
    "sampled rows: dQ without scale": ('out["dq"][r, hs] = scale * (dS @ kv)', 'out["dq"][r, hs] = dS @ kv'),
    "sampled keys: dK without scale": ("dk[c, g] += scale * (dS[:, t] @ qb)", "dk[c, g] += dS[:, t] @ qb"),
    "sampled keys: dV from dS": ("dv[c, g] += P[:, t] @ dob", "dv[c, g] += dS[:, t] @ dob"),
}


def _load(mutated_src):
    mod = types.ModuleType("oracle_mutant")
    exec(compile(mutated_src, "oracle_mutant", "exec"), mod.__dict__)
    return mod


def _pins(orc):
    """A compact battery of the pins in test_oracle_pins.py; raises if any fails."""
    # causal attention (nothing evicted) against SDPA, with gradients
    L, Hq, Hkv, D = 40, 4, 2, 8
    q, k, v, do = (inputs.randn_bf16(s, 900 + i) for i, s in enumerate([(L, Hq, D), (L, Hkv, D), (L, Hkv, D), (L, Hq, D)]))
    scale = 1 / math.sqrt(D)
    res = orc.backward(q, k, v, np.full(L, 1 << 30), scale, do)
    qt, kt, vt = (x.double().clone().requires_grad_(True) for x in (q, k, v))
    o = torch.nn.functional.scaled_dot_product_attention(qt.permute(1, 0, 2)[None], kt.permute(1, 0, 2)[None],
                                                         vt.permute(1, 0, 2)[None], is_causal=True, scale=scale,
                                                         enable_gqa=True)[0].permute(1, 0, 2)
    (o * do.double()).sum().backward()
    np.testing.assert_allclose(res["O"], o.detach().numpy(), rtol=1e-10, atol=1e-10)
    fo, flse = orc.forward(q, k, v, np.full(L, 1 << 30), scale)
    np.testing.assert_allclose(fo, o.detach().numpy(), rtol=1e-10, atol=1e-10)
    for key, g in (("dq", qt.grad), ("dk", kt.grad), ("dv", vt.grad)):
        np.testing.assert_allclose(res[key], g.numpy(), rtol=1e-9, atol=1e-10)
    s = torch.einsum("ihd,jhd->hij", q.double(), k.double().repeat_interleave(Hq // Hkv, dim=1)) * scale
    s = s.masked_fill(~torch.ones(L, L, dtype=torch.bool).tril(), -math.inf)
    np.testing.assert_allclose(res["LSE"], torch.logsumexp(s, dim=-1).numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(flse, torch.logsumexp(s, dim=-1).numpy(), rtol=1e-10, atol=1e-10)
    # replay of the compacted stream (evictions, summaries), with gradients
    L, p, w, s_ = 60, 5, 11, 3
    e = inputs.evict_at_layout(L, p, w, s_, "latest_only")
    q, k, v, do = (inputs.randn_bf16(sh, 950 + i) for i, sh in enumerate([(L, Hq, D), (L, Hkv, D), (L, Hkv, D), (L, Hq, D)]))
    qt, kt, vt = (x.double().clone().requires_grad_(True) for x in (q, k, v))
    O, LSE = stream_sim.replay(qt, kt, vt, p, w, s_, "latest_only", scale)
    (O * do.double()).sum().backward()
    res = orc.backward(q, k, v, e, scale, do)
    np.testing.assert_allclose(res["O"], O.detach().numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(res["LSE"], LSE.detach().numpy(), rtol=1e-10, atol=1e-10)
    for key, g in (("dq", qt.grad), ("dk", kt.grad), ("dv", vt.grad)):
        np.testing.assert_allclose(res[key], g.numpy(), rtol=1e-9, atol=1e-10)
    # the row- and key-sampled forms against the same replay
    pos = np.arange(L)
    rr = orc.rows_reference(q, k, v, e, scale, do, pos)
    np.testing.assert_allclose(rr["O"], O.detach().numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(rr["LSE"], LSE.detach().numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(rr["dq"], qt.grad.numpy(), rtol=1e-9, atol=1e-10)
    sk, sv = orc.keys_reference(q, k, v, e, scale, do, pos)
    np.testing.assert_allclose(sk, kt.grad.numpy(), rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(sv, vt.grad.numpy(), rtol=1e-9, atol=1e-10)


def test_unmutated_oracle_passes_battery():
    _pins(_load(SRC))


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name):
    old, new = MUTATIONS[name]
    assert SRC.count(old) >= 1, f"mutation anchor for {name!r} not found"
    mutant = _load(SRC.replace(old, new))
    with pytest.raises(Exception):
        _pins(mutant)
