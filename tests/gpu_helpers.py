"""Shared helpers of the GPU parity tests."""
import sys

import numpy as np
import torch

# Parity bar for bf16 outputs against the fp64 checker: max |x - x*| and
# ||x - x*||_2 / ||x*||_2 for O, dQ, dK, dV.  LSE (fp32) gets an absolute bound.
MAX_ABS = 2e-2
REL_L2 = 1e-2
LSE_ABS = 1e-3


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


def elementwise_excess(x, ref, base=MAX_ABS):
    """Largest |x - x*| / (base * max(1, |x*|)): <= 1 means every element is
    within ``base`` absolute where |x*| <= 1 and within ``base`` relative above
    (bf16 spacing grows with |x|: rounding an output of magnitude 27 alone
    moves it by up to 0.0625, and P and dS are rounded to bf16 before the
    products, another ~2^-9 |x|)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if x.size == 0:
        return 0.0
    return float((np.abs(x - ref) / (base * np.maximum(1.0, np.abs(ref)))).max())


def assert_close(name, x, ref, max_abs=MAX_ABS, rel_l2=REL_L2, elementwise=True):
    """Parity bar: |x - x*| <= max_abs * max(1, |x*|) per element (plain
    |x - x*| <= max_abs when elementwise is False) and relative L2 <= rel_l2."""
    ma, rl = metrics(x, ref)
    assert np.all(np.isfinite(np.asarray(x, dtype=np.float64))), f"{name}: non-finite values"
    ex = elementwise_excess(x, ref, max_abs) if elementwise else ma / max_abs
    assert ex <= 1.0 and rl <= rel_l2, (f"{name}: maxabs {ma:.3e}, worst error / bound {ex:.3f} (bound "
                                        f"{max_abs} x max(1,|x*|)), relL2 {rl:.3e} (bound {rel_l2})")
    return ma, rl


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def gpu_fwd_bwd(kvs, q, k, v, do, evict_at, scale, cu_seqlens=None, max_seqlen=None, B=None):
    """Run the library on CPU bf16 tensors in packed layout [ntok, H, D]; returns CPU tensors."""
    dev = torch.device("cuda:0")
    qd, kd, vd, dod = (x.to(dev).contiguous() for x in (q, k, v, do))
    ev = torch.from_numpy(np.ascontiguousarray(evict_at, dtype=np.int32)).to(dev)
    if cu_seqlens is None:
        n = q.shape[0]
        B = B or 1
        T = n // B
        shp = lambda x: x.view(B, T, x.shape[1], x.shape[2])
        o, lse = kvs.kvs_evict_attn_fwd(shp(qd), shp(kd), shp(vd), ev.view(B, T), scale)
        dq, dk, dv = kvs.kvs_evict_attn_bwd(shp(dod), shp(qd), shp(kd), shp(vd), o, lse, ev.view(B, T), scale)
        o, dq, dk, dv = (x.reshape(n, x.shape[2], x.shape[3]) for x in (o, dq, dk, dv))
        # [B, Hq, T] -> [Hq, ntok]
        lse = lse.permute(1, 0, 2).reshape(lse.shape[1], n)
    else:
        cu = torch.from_numpy(np.asarray(cu_seqlens, dtype=np.int32)).to(dev)
        o, lse = kvs.kvs_evict_attn_fwd(qd, kd, vd, ev, scale, cu, max_seqlen)
        dq, dk, dv = kvs.kvs_evict_attn_bwd(dod, qd, kd, vd, o, lse, ev, scale, cu, max_seqlen)
    torch.cuda.synchronize()
    return {"O": o.cpu(), "LSE": lse.cpu(), "dq": dq.cpu(), "dk": dk.cpu(), "dv": dv.cpu()}
