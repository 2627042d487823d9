"""Shared helpers of the GPU parity tests."""
import sys

import numpy as np
import torch

# Parity bar for bf16 outputs against the fp64 oracle, per element
#     |x - x*| <= MAX_ABS + ULP_FACTOR * ulp_bf16(x*)                         (O)
#     |x - x*| <= MAX_ABS + ULP_FACTOR * ulp_bf16(x*) + DQ_GAMMA * E           (dQ)
#     |x - x*| <= MAX_ABS + ULP_FACTOR * ulp_bf16(x*) + RSS_LAMBDA * U * S     (dK, dV)
# (ulp_bf16(x*) = spacing of bf16 numbers at x*) and ||x - x*||_2 / ||x*||_2 <= REL_L2.
# Where the bf16 spacing is small the bound is the flat 2e-2; between 8 and 16
# a bf16 output can sit 1/32 from the exact value, which the flat part alone
# cannot allow for.  ULP_FACTOR comes from the CPU model of the kernels'
# roundings (tests/kernel_model.py): at least the model's largest excess over
# the rest of the bound and at most twice it (tests/test_kernel_model.py).
# E = oracle.attention.dq_rounding_scale is the oracle's first-order
# sensitivity of dQ to the bf16 roundings of O (through Delta) and of dS,
# DQ_GAMMA = 2^-8 the relative rounding bound of bf16.  S =
# oracle.attention.dkdv_rounding_rss is the root sum of squares of the terms of
# the dK and dV sums that carry a bf16 rounding (P, dS, O through Delta); the
# roundings of different rows and heads are independent, so the error of such
# a sum stays within RSS_LAMBDA * U * S (U = 2^-8) except with probability at
# most 2 exp(-RSS_LAMBDA^2 / 2) = 5e-11 per element (Hoeffding's inequality,
# as in probabilistic rounding-error analysis).  It matters for large GQA
# groups, whose dK/dV sum G heads; the full-size comparisons (G = 4, 5) omit
# it.  LSE (fp32) gets an absolute bound.
MAX_ABS = 2e-2
REL_L2 = 1e-2
ULP_FACTOR = 0.45
DQ_GAMMA = 2.0 ** -8
RSS_LAMBDA = 7.0
U_BF16 = 2.0 ** -8
LSE_ABS = 1e-3


def ulp_bf16(x):
    """Spacing of bf16 numbers in the binade of |x| (2^(e - 7) for |x| in [2^e, 2^(e+1)))."""
    a = np.maximum(np.abs(np.asarray(x, dtype=np.float64)), 2.0 ** -126)
    return np.exp2(np.floor(np.log2(a)) - 7.0)


def bound(ref, E=None, S=None):
    """Per-element bound of |x - x*| (E: dQ's rounding sensitivity, S: dK's or dV's
    root-sum-square rounding sensitivity; same shape as ref)."""
    b = MAX_ABS + ULP_FACTOR * ulp_bf16(ref)
    if E is not None:
        b = b + DQ_GAMMA * np.asarray(E, dtype=np.float64)
    if S is not None:
        b = b + RSS_LAMBDA * U_BF16 * np.asarray(S, dtype=np.float64)
    return b


def announce(msg: str) -> None:
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def metrics(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = x - ref
    maxabs = float(np.abs(d).max()) if d.size else 0.0
    den = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(d)) / den if den > 0 else float(np.linalg.norm(d))
    return maxabs, rel


def assert_close(name, x, ref, E=None, rel_l2=REL_L2, log=None, extra=None, S=None):
    """Parity bar: |x - x*| <= bound(x*, E, S) (+ ``extra``, roundings a caller adds
    outside the kernels) per element and relative L2 <= rel_l2.
    Returns (flat max |x - x*|, worst |x - x*| / bound, relative L2) and prints them."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert np.all(np.isfinite(x)), f"{name}: non-finite values"
    ma, rl = metrics(x, ref)
    b = bound(ref, E, S) + (0.0 if extra is None else np.asarray(extra, dtype=np.float64))
    ratio = float((np.abs(x - ref) / b).max()) if x.size else 0.0
    line = (f"[parity] {name}: maxabs {ma:.3e} ({'<=' if ma <= MAX_ABS else '>'} {MAX_ABS}) "
            f"worst/bound {ratio:.3f} relL2 {rl:.2e}")
    print(line, flush=True)
    if log is not None:
        log.append((name, ma, ratio, rl))
    assert ratio <= 1.0 and rl <= rel_l2, line
    return ma, ratio, rl


def assert_flat(name, x, ref, max_abs, rel_l2):
    """A special-purpose flat bound (closed forms, single-entry caches)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    ma, rl = metrics(x, ref)
    print(f"[parity] {name}: maxabs {ma:.3e} (bound {max_abs}) relL2 {rl:.2e}", flush=True)
    assert np.all(np.isfinite(x)) and ma <= max_abs and rl <= rel_l2, (name, ma, rl)
    return ma, rl


def assert_lse(name, x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = float(np.abs(x - ref).max()) if x.size else 0.0
    print(f"[parity] {name}: LSE maxabs {err:.2e} (bound {LSE_ABS})", flush=True)
    assert np.all(np.isfinite(x)) and err <= LSE_ABS, f"{name}: LSE error {err}"
    return err


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def gpu_fwd_bwd(kvs, q, k, v, do, evict_at, scale, cu_seqlens=None, max_seqlen=None, B=None, flags=0):
    """Run the library on CPU bf16 tensors in packed layout [ntok, H, D]; returns CPU tensors.
    ``flags`` (kvs.FLAG_*) selects the tile-classifier switches of the *_ex calls."""
    dev = torch.device("cuda:0")
    qd, kd, vd, dod = (x.to(dev).contiguous() for x in (q, k, v, do))
    ev = torch.from_numpy(np.ascontiguousarray(evict_at, dtype=np.int32)).to(dev)
    if cu_seqlens is None:
        n = q.shape[0]
        B = B or 1
        T = n // B
        shp = lambda x: x.view(B, T, x.shape[1], x.shape[2])
        o, lse = kvs.kvs_evict_attn_fwd(shp(qd), shp(kd), shp(vd), ev.view(B, T), scale, flags=flags)
        dq, dk, dv = kvs.kvs_evict_attn_bwd(shp(dod), shp(qd), shp(kd), shp(vd), o, lse, ev.view(B, T), scale,
                                            flags=flags)
        o, dq, dk, dv = (x.reshape(n, x.shape[2], x.shape[3]) for x in (o, dq, dk, dv))
        # [B, Hq, T] -> [Hq, ntok]
        lse = lse.permute(1, 0, 2).reshape(lse.shape[1], n)
    else:
        cu = torch.from_numpy(np.asarray(cu_seqlens, dtype=np.int32)).to(dev)
        o, lse = kvs.kvs_evict_attn_fwd(qd, kd, vd, ev, scale, cu, max_seqlen, flags=flags)
        dq, dk, dv = kvs.kvs_evict_attn_bwd(dod, qd, kd, vd, o, lse, ev, scale, cu, max_seqlen, flags=flags)
    torch.cuda.synchronize()
    return {"O": o.cpu(), "LSE": lse.cpu(), "dq": dq.cpu(), "dk": dk.cpu(), "dv": dv.cpu()}


OUTPUTS = ("O", "LSE", "dq", "dk", "dv")


def assert_switches_bitwise(kvs, base, q, k, v, do, evict_at, scale, cu_seqlens=None, max_seqlen=None, B=None,
                            label=""):
    """The tile-classifier switches (every EMPTY tile processed masked, every FULL
    tile masked) leave every output bit-identical to the plain call ``base``."""
    for flags in (kvs.FLAG_NO_EMPTY_SKIP, kvs.FLAG_FULL_AS_PARTIAL,
                  kvs.FLAG_NO_EMPTY_SKIP | kvs.FLAG_FULL_AS_PARTIAL):
        other = gpu_fwd_bwd(kvs, q, k, v, do, evict_at, scale, cu_seqlens=cu_seqlens, max_seqlen=max_seqlen, B=B,
                            flags=flags)
        for key in OUTPUTS:
            same = torch.equal(base[key].view(torch.int16) if base[key].dtype == torch.bfloat16 else base[key],
                               other[key].view(torch.int16) if other[key].dtype == torch.bfloat16 else other[key])
            assert same, f"{label}: {key} differs bitwise with flags {flags}"
    print(f"[bitwise] {label}: O, LSE, dQ, dK, dV identical under every tile-classifier switch", flush=True)
