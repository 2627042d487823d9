"""fp64 decode attention over the live entries of a streamed KV cache (test infrastructure).

Section 2 ("KV-streams") evicts keys and values directly in the inference
engine's cache; nothing evicted comes back, and the query generated at
trace position t attends over exactly the entries live at that moment.  With
the trainer's eviction indices (one e_j per key: key j is deleted when token
e_j is generated) that live set is

    R(t) = { j : j <= t  and  e_j > t },

the keys that row t of the eviction-masked attention sees.  For q-head h of
KV head g = h // (Hq // Hkv):

    s_j  = scale * <q^h, k_j^g>          for j in R
    LSE  = ln sum_{j in R} exp(s_j)
    O    = sum_{j in R} exp(s_j - LSE) v_j^g

written out directly (two-pass softmax, fp64).  The order of the entries in
the cache does not matter.  An empty live set gives O = 0 and LSE = -inf.
Test infrastructure only; shares no code with the HIP path.
"""
from __future__ import annotations

import numpy as np


def live_set(evict_at, t: int) -> np.ndarray:
    """Trace positions live in the cache when token t is generated: j <= t with e_j > t."""
    e = np.asarray(evict_at, dtype=np.int64)[: t + 1]
    return np.nonzero(e > t)[0]


def _f64(x) -> np.ndarray:
    """Exact widening of numpy arrays or torch tensors (bf16 included) to fp64."""
    if hasattr(x, "detach"):
        return x.detach().to("cpu").double().numpy()
    return np.asarray(x, dtype=np.float64)


def decode(q, k, v, live, scale: float):
    """One query token: q [Hq, D], k/v [N, Hkv, D] (numpy or torch, any float),
    live = indices into k/v.  Returns O [Hq, D] and LSE [Hq] in fp64.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    live = np.asarray(live, dtype=np.int64)
    Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    O = np.zeros((Hq, D))
    LSE = np.full(Hq, -np.inf)
    if live.size == 0:
        return O, LSE
    for h in range(Hq):
        g = h // G
        s = scale * (k[live, g, :] @ q[h])
        m = s.max()
        w = np.exp(s - m)
        tot = w.sum()
        O[h] = (w / tot) @ v[live, g, :]
        LSE[h] = m + np.log(tot)
    return O, LSE
