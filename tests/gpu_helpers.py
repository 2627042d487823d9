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


def scaled_max_abs(ref, base=MAX_ABS):
    """Absolute bound for outputs whose magnitude exceeds 1 (short traces, where a
    key is seen by few queries and dV sums G heads of dO with P near 1): bf16
    spacing grows with |x|, so the bound grows with max|x*|.  Equals ``base``
    when max|x*| <= 1."""
    return base * max(1.0, float(np.abs(np.asarray(ref)).max(initial=0.0)))


def assert_close(name, x, ref, max_abs=MAX_ABS, rel_l2=REL_L2):
    ma, rl = metrics(x, ref)
    assert np.all(np.isfinite(np.asarray(x, dtype=np.float64))), f"{name}: non-finite values"
    assert ma <= max_abs and rl <= rel_l2, f"{name}: maxabs {ma:.3e} (bound {max_abs}), relL2 {rl:.3e} (bound {rel_l2})"
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
