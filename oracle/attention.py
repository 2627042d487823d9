"""fp64 eviction-masked attention: the definition, written out (test infrastructure).

Section 2 ("KV-streams") keeps every retained key and value at its original
position and replaces the deletion of a span by an attention mask in a single
pass over the continuous trace; the engine drops evicted keys and values for
good and the trainer mirrors the drop with a mask (Section 7, second
paragraph), so each key ``j`` of a trace has one eviction index ``e_j`` and
query ``i`` attends to it iff

    j <= i < e_j            (any e_j >= L means "never evicted").

For one trace of length L, q-head h and its KV head g = h // (Hq // Hkv):

    V(i)    = { j : j <= i < min(e_j, L) }
    s_ij    = scale * <q_i^h, k_j^g>
    LSE_i   = ln sum_{j in V(i)} exp(s_ij)
    P_ij    = exp(s_ij - LSE_i)  on V(i), else 0
    O_i     = sum_j P_ij v_j^g

and for the scalar loss sum(dO * O):

    dP_ij   = <dO_i, v_j^g>
    Delta_i = sum_j P_ij dP_ij
    dS_ij   = P_ij (dP_ij - Delta_i)
    dQ_i    = scale sum_j dS_ij k_j^g
    dK_j^g  = scale sum_{h in g} sum_i dS_ij q_i^h
    dV_j^g  = sum_{h in g} sum_i P_ij dO_i^h

The mask is built explicitly as a boolean matrix; the softmax is two-pass
(row max, then sum) over the full causal prefix of each block of query rows.
Nothing is skipped.  Inputs are the exact bf16 values widened to fp64.
For traces too long for that, ``rows_reference`` and ``keys_reference``
evaluate the same definitions at chosen rows or keys, each row over its
visible set V(i) gathered from ``evict_at``.

Parity of every function here is pinned by tests against causal attention
(``e = inf``), a brute-force stream replay, finite differences, closed forms
and hand counts; see the module ``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

import numpy as np

ROW_BLOCK = 256


def _f64(x) -> np.ndarray:
    if hasattr(x, "detach"):  # torch tensor (bf16 or float)
        import torch

        return x.detach().to(torch.float64).cpu().numpy()
    return np.asarray(x, dtype=np.float64)


def visible_mask(e: np.ndarray, L: int, i0: int, i1: int, j1: int) -> np.ndarray:
    """Boolean mask of rows ``[i0, i1)`` by columns ``[0, j1)``: ``j <= i < min(e_j, L)``."""
    i = np.arange(i0, i1)[:, None]
    j = np.arange(0, j1)[None, :]
    ej = np.minimum(e[:j1].astype(np.int64), L)[None, :]
    return (j <= i) & (i < ej)


def check_evict_at(e: np.ndarray, L: int) -> None:
    """Every key must be visible to itself: ``e_j > j``."""
    e = np.asarray(e, dtype=np.int64)
    if e.shape != (L,):
        raise ValueError(f"evict_at has shape {e.shape}, expected ({L},)")
    bad = np.nonzero(e <= np.arange(L))[0]
    if bad.size:
        raise ValueError(f"evict_at[{bad[0]}] = {e[bad[0]]} <= {bad[0]}")


def _trace_forward(q, k, v, e, scale):
    """One trace: q [L,Hq,D], k/v [L,Hkv,D] fp64, e [L]. Returns O [L,Hq,D], LSE [Hq,L]."""
    L, Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    O = np.zeros((L, Hq, v.shape[2]))
    LSE = np.zeros((Hq, L))
    for h in range(Hq):
        g = h // G
        for i0 in range(0, L, ROW_BLOCK):
            i1 = min(i0 + ROW_BLOCK, L)
            M = visible_mask(e, L, i0, i1, i1)
            S = scale * (q[i0:i1, h, :] @ k[:i1, g, :].T)
            S = np.where(M, S, -np.inf)
            m = S.max(axis=1, keepdims=True)
            E = np.where(M, np.exp(S - m), 0.0)
            l = E.sum(axis=1, keepdims=True)
            P = E / l
            O[i0:i1, h, :] = P @ v[:i1, g, :]
            LSE[h, i0:i1] = (m + np.log(l))[:, 0]
    return O, LSE


def _trace_backward(q, k, v, e, scale, do):
    """One trace: returns O, LSE, Delta [Hq,L], dQ, dK, dV (fp64)."""
    L, Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    O = np.zeros((L, Hq, v.shape[2]))
    LSE = np.zeros((Hq, L))
    Delta = np.zeros((Hq, L))
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for h in range(Hq):
        g = h // G
        for i0 in range(0, L, ROW_BLOCK):
            i1 = min(i0 + ROW_BLOCK, L)
            M = visible_mask(e, L, i0, i1, i1)
            S = scale * (q[i0:i1, h, :] @ k[:i1, g, :].T)
            S = np.where(M, S, -np.inf)
            m = S.max(axis=1, keepdims=True)
            E = np.where(M, np.exp(S - m), 0.0)
            l = E.sum(axis=1, keepdims=True)
            P = E / l
            O[i0:i1, h, :] = P @ v[:i1, g, :]
            LSE[h, i0:i1] = (m + np.log(l))[:, 0]
            dP = do[i0:i1, h, :] @ v[:i1, g, :].T
            dlt = (P * dP).sum(axis=1, keepdims=True)
            Delta[h, i0:i1] = dlt[:, 0]
            dS = P * (dP - dlt)
            dq[i0:i1, h, :] = scale * (dS @ k[:i1, g, :])
            dk[:i1, g, :] += scale * (dS.T @ q[i0:i1, h, :])
            dv[:i1, g, :] += P.T @ do[i0:i1, h, :]
    return O, LSE, Delta, dq, dk, dv


def _split(cu_seqlens, n):
    if cu_seqlens is None:
        return [(0, n)]
    cu = [int(c) for c in cu_seqlens]
    return [(cu[b], cu[b + 1]) for b in range(len(cu) - 1)]


def forward(q, k, v, evict_at, scale, cu_seqlens=None):
    """Packed traces ``[ntok, H, D]`` (``cu_seqlens`` = trace offsets; None = one trace).

    ``evict_at`` is trace-local.  Returns fp64 ``O [ntok,Hq,D]`` and ``LSE [Hq,ntok]``.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    e = np.asarray(evict_at, dtype=np.int64)
    n, Hq, _ = q.shape
    if k.shape[0] != n or v.shape[0] != n or e.shape != (n,) or Hq % k.shape[1]:
        raise ValueError("shape mismatch")
    O = np.zeros((n, Hq, v.shape[2]))
    LSE = np.zeros((Hq, n))
    for a, b in _split(cu_seqlens, n):
        if b == a:
            continue
        check_evict_at(e[a:b], b - a)
        O[a:b], LSE[:, a:b] = _trace_forward(q[a:b], k[a:b], v[a:b], e[a:b], scale)
    return O, LSE


def backward(q, k, v, evict_at, scale, do, cu_seqlens=None):
    """Gradients of ``sum(do * O)``; returns dict with O, LSE, Delta, dq, dk, dv (fp64)."""
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    e = np.asarray(evict_at, dtype=np.int64)
    n, Hq, _ = q.shape
    if k.shape[0] != n or v.shape[0] != n or e.shape != (n,) or do.shape != (n, Hq, v.shape[2]):
        raise ValueError("shape mismatch")
    out = {
        "O": np.zeros((n, Hq, v.shape[2])),
        "LSE": np.zeros((Hq, n)),
        "Delta": np.zeros((Hq, n)),
        "dq": np.zeros_like(q),
        "dk": np.zeros_like(k),
        "dv": np.zeros_like(v),
    }
    for a, b in _split(cu_seqlens, n):
        if b == a:
            continue
        check_evict_at(e[a:b], b - a)
        O, LSE, Dl, dq, dk, dv = _trace_backward(q[a:b], k[a:b], v[a:b], e[a:b], scale, do[a:b])
        out["O"][a:b], out["LSE"][:, a:b], out["Delta"][:, a:b] = O, LSE, Dl
        out["dq"][a:b], out["dk"][a:b], out["dv"][a:b] = dq, dk, dv
    return out


def visible_pairs(evict_at, lengths) -> int:
    """Visible (query, key) pairs per head, counted from the explicit mask row by row."""
    e = np.asarray(evict_at, dtype=np.int64)
    tot, off = 0, 0
    for L in lengths:
        for i0 in range(0, L, ROW_BLOCK):
            i1 = min(i0 + ROW_BLOCK, L)
            tot += int(visible_mask(e[off:off + L], L, i0, i1, i1).sum())
        off += L
    return tot


def dq_rounding_scale(q, k, v, evict_at, scale, do, rows, cu_seqlens=None):
    """Sensitivity of dQ to the two roundings every bf16 backward makes before its dQ sum.

    A backward that receives O in bf16 forms ``Delta_i`` from the rounded O, and
    a bf16 matrix-core product rounds every ``dS_ij`` to bf16 before
    ``dQ_i = scale sum_j dS_ij k_j``.  A relative error of at most u in each
    ``O_id`` and in each ``dS_ij`` moves ``dQ_id`` by at most ``u`` times

        E_id = scale * ( sum_j |dS_ij| |k_jd|  +  |sum_j P_ij k_jd| * sum_d' |dO_id'| |O_id'| )

    (first order; the second term through ``dS_ij = P_ij (dP_ij - Delta_i)``).
    Returns ``E`` (fp64) for the packed query rows ``rows``: shape
    ``[len(rows), Hq, D]``.  Test infrastructure for tolerances: P, dS and O
    are the exact quantities of the definition above, row by row.
    """
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    e = np.asarray(evict_at, dtype=np.int64)
    rows = np.asarray(rows, dtype=np.int64)
    n, Hq, D = q.shape
    G = Hq // k.shape[1]
    out = np.zeros((rows.size, Hq, D))
    for a, b in _split(cu_seqlens, n):
        sel = np.nonzero((rows >= a) & (rows < b))[0]
        if sel.size == 0:
            continue
        L = b - a
        for c0 in range(0, sel.size, ROW_BLOCK):
            idx = sel[c0:c0 + ROW_BLOCK]
            il = rows[idx] - a                       # trace-local rows of this block
            j1 = int(il.max()) + 1
            ej = np.minimum(e[a:a + j1], L)[None, :]
            jj = np.arange(j1)[None, :]
            M = (jj <= il[:, None]) & (il[:, None] < ej)
            for h in range(Hq):
                g = h // G
                S = np.where(M, scale * (q[a + il, h, :] @ k[a:a + j1, g, :].T), -np.inf)
                E = np.where(M, np.exp(S - S.max(axis=1, keepdims=True)), 0.0)
                P = E / E.sum(axis=1, keepdims=True)
                dP = do[a + il, h, :] @ v[a:a + j1, g, :].T
                dlt = (P * dP).sum(axis=1, keepdims=True)
                dS = P * (dP - dlt)
                O = P @ v[a:a + j1, g, :]
                R = (np.abs(do[a + il, h, :]) * np.abs(O)).sum(axis=1, keepdims=True)
                out[idx, h, :] = scale * (np.abs(dS) @ np.abs(k[a:a + j1, g, :])
                                          + np.abs(P @ k[a:a + j1, g, :]) * R)
    return out


def dkdv_rounding_rss(q, k, v, evict_at, scale, do, cu_seqlens=None):
    """Root-sum-square sensitivity of dK and dV to the roundings every bf16 backward makes.

    ``dV_jd = sum_{h in g} sum_i P_hij dO_hid`` takes P rounded to bf16, and
    ``dK_jd = scale sum_{h in g} sum_i dS_hij q_hid`` takes dS rounded to bf16,
    with ``dS_hij = P_hij (dP_hij - Delta_hi)`` and ``Delta_hi`` formed from the
    bf16 O.  Each rounding is a relative error of at most u, and the sums run
    over many rows and heads whose roundings are independent, so the error of
    a sum is of the order of u times the root sum of squares of its terms
    (probabilistic rounding-error analysis, Higham and Mary, SIAM J. Sci.
    Comput. 41(5), 2019), not u times the sum of their magnitudes:

        SV_jd = sqrt( sum_{h in g} sum_i (P_hij dO_hid)^2 )
        SK_jd = scale * sqrt( sum_{h in g} sum_i ( dS_hij^2 + (P_hij R_hi)^2 ) q_hid^2 ),
        R_hi  = sqrt( sum_d' (dO_hid' O_hid')^2 )   (the rounding of O reaching Delta)

    (g: the KV head of key j; i over the rows that see key j).  Returns
    ``(SK, SV)`` (fp64), each shaped like k.  Test infrastructure for
    tolerances: P, dS and O are the exact quantities of the definitions above.
    """
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    e = np.asarray(evict_at, dtype=np.int64)
    n, Hq, D = q.shape
    G = Hq // k.shape[1]
    SK2 = np.zeros_like(k)
    SV2 = np.zeros_like(v)
    for a, b in _split(cu_seqlens, n):
        L = b - a
        if L == 0:
            continue
        for i0 in range(0, L, ROW_BLOCK):
            i1 = min(i0 + ROW_BLOCK, L)
            M = visible_mask(e[a:b], L, i0, i1, i1)
            for h in range(Hq):
                g = h // G
                S = np.where(M, scale * (q[a + i0:a + i1, h, :] @ k[a:a + i1, g, :].T), -np.inf)
                m = S.max(axis=1, keepdims=True)
                E = np.where(M, np.exp(S - m), 0.0)
                P = E / E.sum(axis=1, keepdims=True)
                dP = do[a + i0:a + i1, h, :] @ v[a:a + i1, g, :].T
                dlt = (P * dP).sum(axis=1, keepdims=True)
                dS = P * (dP - dlt)
                O = P @ v[a:a + i1, g, :]
                R2 = ((do[a + i0:a + i1, h, :] * O) ** 2).sum(axis=1, keepdims=True)
                SV2[a:a + i1, g, :] += (P ** 2).T @ (do[a + i0:a + i1, h, :] ** 2)
                SK2[a:a + i1, g, :] += (dS ** 2 + P ** 2 * R2).T @ (q[a + i0:a + i1, h, :] ** 2)
    return scale * np.sqrt(SK2), np.sqrt(SV2)


def _gatherable(x):
    """A numpy array to gather rows from without widening the whole tensor: the
    raw 16-bit patterns of a bf16 torch tensor (no copy), else fp64."""
    if hasattr(x, "detach"):
        import torch

        if x.dtype == torch.bfloat16:
            return x.detach().cpu().contiguous().view(torch.int16).numpy()
    return _f64(x)


def _widen(a: np.ndarray) -> np.ndarray:
    """fp64 values of elements gathered from ``_gatherable``: its int16 arrays
    hold bf16 bit patterns, which become the fp32 with those upper 16 bits
    (exact), widened to fp64; floats are widened."""
    if a.dtype == np.int16:
        return (a.astype(np.int32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float64)


def _visible_keys(e_tr: np.ndarray, L: int, i: int) -> np.ndarray:
    """Trace-local keys of V(i) = { j <= i : i < min(e_j, L) }, ascending."""
    return np.nonzero(np.minimum(e_tr[:i + 1], L) > i)[0]


def _trace_of(pos: int, cu_seqlens, n: int):
    for a, b in _split(cu_seqlens, n):
        if a <= pos < b:
            return a, b
    raise ValueError(f"position {pos} outside [0, {n})")


def rows_reference(q, k, v, evict_at, scale, do, rows, cu_seqlens=None):
    """O, LSE, Delta, dQ and the dQ rounding sensitivity E at the packed query rows ``rows`` only.

    Each row's quantities depend on its own visible set V(i) alone, so they are
    computed from that set (gathered from ``evict_at``) instead of the full
    causal prefix, for the G q-heads of a KV head together: the same
    definitions as ``backward`` and ``dq_rounding_scale`` at any trace length.
    Only the gathered rows and keys are widened to fp64.  Returns fp64
    ``O, dq, E [len(rows), Hq, D]`` and ``LSE, Delta [Hq, len(rows)]``.
    """
    e = np.asarray(evict_at, dtype=np.int64)
    rows = np.asarray(rows, dtype=np.int64)
    n, Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    out = {"O": np.zeros((rows.size, Hq, D)), "dq": np.zeros((rows.size, Hq, D)), "E": np.zeros((rows.size, Hq, D)),
           "LSE": np.zeros((Hq, rows.size)), "Delta": np.zeros((Hq, rows.size))}
    qr, kr, vr, dor = (_gatherable(x) for x in (q, k, v, do))
    for a, b in _split(cu_seqlens, n):
        check_evict_at(e[a:b], b - a)
    for r, pos in enumerate(rows):
        a, b = _trace_of(int(pos), cu_seqlens, n)
        js = a + _visible_keys(e[a:b], b - a, int(pos) - a)
        for g in range(Hkv):
            hs = slice(g * G, (g + 1) * G)
            kv, vv = _widen(kr[js, g]), _widen(vr[js, g])          # [|V(i)|, D]
            qg, dog = _widen(qr[pos, hs]), _widen(dor[pos, hs])    # [G, D]
            S = scale * (qg @ kv.T)
            m = S.max(axis=1, keepdims=True)
            ex = np.exp(S - m)
            l = ex.sum(axis=1, keepdims=True)
            P = ex / l
            O = P @ vv
            dP = dog @ vv.T
            dlt = (P * dP).sum(axis=1, keepdims=True)
            dS = P * (dP - dlt)
            out["O"][r, hs], out["LSE"][hs, r], out["Delta"][hs, r] = O, (m + np.log(l))[:, 0], dlt[:, 0]
            out["dq"][r, hs] = scale * (dS @ kv)
            R = (np.abs(dog) * np.abs(O)).sum(axis=1, keepdims=True)
            out["E"][r, hs] = scale * (np.abs(dS) @ np.abs(kv) + np.abs(P @ kv) * R)
    return out


def keys_reference(q, k, v, evict_at, scale, do, keys, cu_seqlens=None):
    """dK and dV at the packed keys ``keys`` only.

    Key j of a trace is seen by the rows R(j) = [j, min(e_j, L)).  The union
    of those rows is processed once, in blocks of consecutive rows as in
    ``backward`` (no block spans a gap), but each block's columns are only
    the keys some row of the block can see (j <= the block's last row,
    min(e_j, L) > its first), with the explicit mask on top: every row's P
    and dS, so its LSE and Delta, are those of the definition.  The G q-heads
    of a KV head are stacked as extra rows.  Returns fp64
    ``dk, dv [len(keys), Hkv, D]``.
    """
    e = np.asarray(evict_at, dtype=np.int64)
    keys = np.asarray(keys, dtype=np.int64)
    n, Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    dk = np.zeros((keys.size, Hkv, D))
    dv = np.zeros((keys.size, Hkv, D))
    qr, kr, vr, dor = (_gatherable(x) for x in (q, k, v, do))
    for a, b in _split(cu_seqlens, n):
        L = b - a
        mine = np.nonzero((keys >= a) & (keys < b))[0]
        if mine.size == 0:
            continue
        check_evict_at(e[a:b], L)
        et = np.minimum(e[a:b], L)
        rows = np.unique(np.concatenate([np.arange(keys[c] - a, et[keys[c] - a]) for c in mine]))
        runs = np.split(rows, np.nonzero(np.diff(rows) > 1)[0] + 1)   # consecutive rows
        blocks = [r[c0:c0 + ROW_BLOCK] for r in runs for c0 in range(0, r.size, ROW_BLOCK)]
        for il in blocks:
            cand = np.nonzero(et[:il[-1] + 1] > il[0])[0]          # keys some row of the block may see
            M = (cand[None, :] <= il[:, None]) & (il[:, None] < et[cand][None, :])
            M = np.repeat(M, G, axis=0)                           # rows (i, h) with h the fast index
            pos = {int(j): t for t, j in enumerate(cand)}
            cols = [(c, pos[int(keys[c] - a)]) for c in mine if int(keys[c] - a) in pos]
            if not cols:
                continue
            for g in range(Hkv):
                hs = slice(g * G, (g + 1) * G)
                qb = _widen(qr[a + il, hs]).reshape(-1, D)
                dob = _widen(dor[a + il, hs]).reshape(-1, D)
                kc, vc = _widen(kr[a + cand, g]), _widen(vr[a + cand, g])
                S = np.where(M, scale * (qb @ kc.T), -np.inf)
                E = np.where(M, np.exp(S - S.max(axis=1, keepdims=True)), 0.0)
                P = E / E.sum(axis=1, keepdims=True)
                dP = dob @ vc.T
                dS = P * (dP - (P * dP).sum(axis=1, keepdims=True))
                for c, t in cols:
                    dv[c, g] += P[:, t] @ dob
                    dk[c, g] += scale * (dS[:, t] @ qb)
    return dk, dv
