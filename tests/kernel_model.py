"""CPU model of the HIP kernels' arithmetic (test infrastructure, not the oracle).

The fp64 oracle in ``oracle/`` defines what the library computes.  This
module replays, in numpy, the precision choices the gfx950 kernels make on the
way there, so that the tests can tell how far a kernel with exactly these
roundings lies from the exact result, and so derive the parity bound from the
number formats instead of guessing it:

* forward: scores ``S = Q K^T`` in fp32 (exact bf16 products, fp32 sums);
  per wave of 32 query rows, key sub-tiles of 32 (D = 128) or 64 (D = 64) keys
  in increasing order; an online softmax in base 2 whose reference maximum only
  moves when some row of the wave sees a tile maximum more than 8 above its
  own (one decision for the whole wave); ``P = exp2(S * scale * log2 e - m)``
  in fp32, rounded to bf16 before the ``P V`` product, fp32 accumulation; the
  row sum from the fp32 ``P``; ``O = bf16(acc * (1 / l))`` and
  ``LSE = (m + log2 l) ln 2`` in fp32;
* backward preprocess: ``Delta = sum(O_bf16 * dO)`` in fp32 and
  ``LSE * log2 e`` in fp32;
* dK/dV kernel: ``P = exp2(S * scale * log2 e - LSE * log2 e)`` in fp32,
  rounded to bf16 for ``dV += P^T dO`` and to fp16 for
  ``dS = P (dP - Delta)`` (fp32 product, rounded to bf16), ``dK += dS^T Q``;
  outputs ``bf16(dV)``, ``bf16(dK * scale)``;
* dQ kernel: the same fp32 ``P`` unrounded, ``dS = bf16(P (dP - Delta))``,
  ``dQ = bf16((dS K) * scale)``.

Every fp32 step is modelled as the exact (fp64) result rounded once to fp32
(the kernels' own summation orders differ; that difference is far below the
bf16 roundings modelled here).  The mask is the eviction mask of Section 2
("KV-streams"): query i sees key j iff ``j <= i < evict_at[j]``.
"""
from __future__ import annotations

import math

import numpy as np

LOG2E = 1.4426950408889634
LN2 = 0.6931471805599453


def f32(x):
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def bf16(x):
    """Round to bf16 (nearest even) and widen back to fp64; inf and nan pass through."""
    a = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)
    out = r.view(np.float32).astype(np.float64)
    special = ~np.isfinite(a)
    if special.any():
        out = np.where(special, a.astype(np.float64), out)
    return out


def f16(x):
    return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


def ulp_bf16(x):
    """Spacing of bf16 numbers in the binade of |x| (2^(e - 7) for |x| in [2^e, 2^(e+1)))."""
    a = np.maximum(np.abs(np.asarray(x, dtype=np.float64)), 2.0 ** -126)
    return np.exp2(np.floor(np.log2(a)) - 7.0)


def _mask(e, L, rows, cols):
    ej = np.minimum(np.asarray(e, dtype=np.int64)[cols], L)
    return (cols[None, :] <= rows[:, None]) & (rows[:, None] < ej[None, :])


def forward_trace(q, k, v, e, scale, guard=True):
    """One trace: q [L,Hq,D], k/v [L,Hkv,D] (bf16 values as fp64), e [L].

    Returns O [L,Hq,D] (bf16 values) and LSE [Hq,L] (fp32 values).  All waves
    (32-row blocks) advance together, one key sub-tile at a time; each wave's
    rescale decision is taken over its own rows only.  A wave to which a
    sub-tile is EMPTY takes it fully masked, which leaves its state unchanged
    (no row can trigger, every P is 0), exactly as skipping it does, so only
    rows with a visible key in the sub-tile are updated.  With
    ``guard=False`` the rescale factor of a row that has seen no visible key
    is exp2(-inf - -inf), as in a kernel without the guard."""
    L, Hq, D = q.shape
    G = Hq // k.shape[1]
    BN = 32 if D == 128 else 64
    sl2 = float(np.float32(scale * LOG2E))
    Lp = -(-L // 32) * 32
    rows_all = np.arange(Lp)
    O = np.zeros((L, Hq, D))
    LSE = np.zeros((Hq, L))
    e = np.asarray(e, dtype=np.int64)
    for h in range(Hq):
        g = h // G
        S_all = f32(q[:, h] @ k[:, g].T)
        m = np.full(Lp, -np.inf)
        l = np.zeros(Lp)
        acc = np.zeros((Lp, D))
        with np.errstate(invalid="ignore", over="ignore"):
            for j0 in range(0, L, BN):
                r0 = (j0 // 32) * 32            # first wave that can see this sub-tile
                rows = rows_all[r0:]
                cols = np.arange(j0, min(j0 + BN, L))
                vis = _mask(e, L, rows, cols) & (rows < L)[:, None]
                s = np.full((rows.size, cols.size), -np.inf)
                ok = rows < L
                s[ok] = np.where(vis[ok], S_all[np.ix_(rows[ok], cols)], -np.inf)
                mx = f32(s.max(axis=1) * sl2)
                mr = m[r0:]
                trig = np.repeat((mx > mr + 8.0).reshape(-1, 32).any(axis=1), 32)
                t = np.nonzero(trig)[0]            # rows of the waves whose reference maximum moves
                if t.size:
                    m_new = np.maximum(mr[t], mx[t])
                    if guard:
                        alpha = np.where(m_new == mr[t], 1.0, f32(np.exp2(mr[t] - m_new)))
                    else:
                        alpha = f32(np.exp2(mr[t] - m_new))
                    l[r0 + t] = f32(l[r0 + t] * alpha)
                    acc[r0 + t] = f32(acc[r0 + t] * alpha[:, None])
                    m[r0 + t] = m_new
                a_ = np.nonzero(vis.any(axis=1))[0]   # rows with a visible key here (P = 0 elsewhere)
                if a_.size:
                    mu = m[r0 + a_]
                    m_use = np.where(mu == -np.inf, 0.0, mu)
                    p = f32(np.exp2(f32(s[a_] * sl2 - m_use[:, None])))
                    l[r0 + a_] = f32(l[r0 + a_] + p.sum(axis=1))
                    acc[r0 + a_] = f32(acc[r0 + a_] + bf16(p) @ v[cols, g])
            inv = f32(1.0 / l[:L])
            O[:, h] = bf16(f32(acc[:L] * inv[:, None]))
            LSE[h] = f32((m[:L] + np.log2(l[:L])) * LN2)
    return O, LSE


def backward_trace(q, k, v, e, scale, do, O, LSE):
    """One trace, given the forward's bf16 O and fp32 LSE: returns dQ, dK, dV (bf16 values)."""
    L, Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    sl2 = float(np.float32(scale * LOG2E))
    rows = np.arange(L)
    vis = _mask(e, L, rows, rows)
    delta = f32((O * do).sum(axis=2))                # [L, Hq]
    lse2 = f32(LSE * LOG2E)                          # [Hq, L]
    dq = np.zeros_like(q)
    dk_acc = np.zeros_like(k)
    dv_acc = np.zeros_like(v)
    for h in range(Hq):
        g = h // G
        x = f32(f32(q[:, h] @ k[:, g].T) * sl2 - lse2[h][:, None])
        P = np.where(vis, f32(np.exp2(np.where(vis, x, 0.0))), 0.0)
        dP = f32(do[:, h] @ v[:, g].T - delta[:, h][:, None])
        dv_acc[:, g] = f32(dv_acc[:, g] + bf16(P).T @ do[:, h])
        dk_acc[:, g] = f32(dk_acc[:, g] + bf16(f32(f16(P) * dP)).T @ q[:, h])
        dq[:, h] = bf16(f32(f32(bf16(f32(P * dP)) @ k[:, g]) * scale))
    return dq, bf16(f32(dk_acc * scale)), bf16(dv_acc)


def run(q, k, v, e, scale, do, cu_seqlens=None, guard=True):
    """Packed traces [ntok, H, D] (cu_seqlens = offsets; None = one trace): dict of O, LSE, dq, dk, dv."""
    q, k, v, do = (np.asarray(x, dtype=np.float64) for x in (q, k, v, do))
    e = np.asarray(e, dtype=np.int64)
    n = q.shape[0]
    cu = [0, n] if cu_seqlens is None else [int(c) for c in cu_seqlens]
    out = {"O": np.zeros_like(q), "LSE": np.zeros((q.shape[1], n)), "dq": np.zeros_like(q),
           "dk": np.zeros_like(k), "dv": np.zeros_like(v)}
    for a, b in zip(cu[:-1], cu[1:]):
        if b == a:
            continue
        O, LSE = forward_trace(q[a:b], k[a:b], v[a:b], e[a:b], scale, guard=guard)
        out["O"][a:b], out["LSE"][:, a:b] = O, LSE
        if np.isfinite(O).all():
            dq, dk, dv = backward_trace(q[a:b], k[a:b], v[a:b], e[a:b], scale, do[a:b], O, LSE)
            out["dq"][a:b], out["dk"][a:b], out["dv"][a:b] = dq, dk, dv
        else:
            for key in ("dq", "dk", "dv"):
                out[key][a:b] = np.nan
    return out


def excess_ulps(x, ref, flat=2e-2):
    """max over elements of max(0, |x - x*| - flat) / ulp_bf16(x*)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if x.size == 0:
        return 0.0
    return float((np.maximum(np.abs(x - ref) - flat, 0.0) / ulp_bf16(ref)).max())


def math_check():
    """Sanity of the rounding helpers against numbers whose bf16 / fp16 forms are known."""
    assert bf16(1.0 + 2.0 ** -8) == 1.0            # tie -> even
    assert bf16(1.0 + 3 * 2.0 ** -9) == 1.0 + 2.0 ** -7
    assert f16(1.0 + 2.0 ** -11) == 1.0
    assert ulp_bf16(27.0) == 0.125 and ulp_bf16(1.0) == 2.0 ** -7 and ulp_bf16(0.75) == 2.0 ** -8
    assert math.isnan(float(bf16(np.nan))) and bf16(-np.inf) == -np.inf
