"""Guard bands around every buffer the library writes (MI355X).

Each output (O, LSE, dQ, dK, dV, the paged decode's O and LSE) and each
workspace sits inside a larger allocation whose bytes before and after it hold
a fixed pattern; the calls go straight through the C ABI.  After the calls
every guard byte must be unchanged (no write outside the caller's buffers,
however the grid and the trace tails line up), and the outputs must equal,
bit for bit, those of the same calls on ordinary allocations (results do not
depend on where buffers sit).  Every case prints its name before it runs.
"""
import ctypes
import math

import numpy as np
import pytest
import torch

from paper_2609_35750_amd import inputs
from tests.gpu_helpers import announce

pytestmark = pytest.mark.gpu

GUARD = 4096       # bytes on each side (keeps 256-byte alignment for workspaces)
PATTERN = 0x5B


@pytest.fixture(scope="module")
def kvs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35750_amd import kvs as k

    return k


class Banded:
    """A tensor view of `nbytes` inside an allocation with guard bands on both sides."""

    def __init__(self, shape, dtype, dev):
        n = int(np.prod(shape)) if len(shape) else 1
        nbytes = n * torch.empty((), dtype=dtype).element_size()
        self.buf = torch.full((GUARD + nbytes + GUARD,), PATTERN, dtype=torch.uint8, device=dev)
        self.t = self.buf[GUARD:GUARD + nbytes].view(dtype).view(shape)
        self.nbytes = nbytes

    def guards_intact(self):
        b = self.buf.cpu().numpy()
        return bool(np.all(b[:GUARD] == PATTERN) and np.all(b[GUARD + self.nbytes:] == PATTERN))


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _run(kvs, q, k, v, do, ev, cu, B, T, ntok, Hq, Hkv, D, scale, banded):
    """Forward + backward through the C ABI; outputs and workspaces banded or plain."""
    dev = q.device
    lib = kvs.lib

    def alloc(shape, dt):
        return Banded(shape, dt, dev) if banded else torch.empty(shape, dtype=dt, device=dev)

    def tens(x):
        return x.t if banded else x

    lse_shape = (Hq, ntok) if cu is not None else (B, Hq, T)
    o, lse = alloc(tuple(q.shape), torch.bfloat16), alloc(lse_shape, torch.float32)
    dq, dk, dv = alloc(tuple(q.shape), torch.bfloat16), alloc(tuple(k.shape), torch.bfloat16), \
        alloc(tuple(k.shape), torch.bfloat16)
    if cu is None:
        nf = lib.kvs_evict_attn_fwd_workspace(B, T, Hq, Hkv, D)
        nb = lib.kvs_evict_attn_bwd_workspace(B, T, Hq, Hkv, D)
    else:
        mx = int(torch.diff(cu).max().item())
        nf = lib.kvs_evict_attn_varlen_fwd_workspace(B, ntok, mx, Hq, Hkv, D)
        nb = lib.kvs_evict_attn_varlen_bwd_workspace(B, ntok, mx, Hq, Hkv, D)
    wf, wb = alloc((max(nf, 1),), torch.uint8), alloc((max(nb, 1),), torch.uint8)
    if cu is None:
        st = lib.kvs_evict_attn_fwd(_p(q), _p(k), _p(v), _p(ev), _p(tens(o)), _p(tens(lse)), B, T, Hq, Hkv, D, scale,
                                    _p(tens(wf)), nf, _stream())
        assert st == 0, kvs.lib.kvs_last_error()
        st = lib.kvs_evict_attn_bwd(_p(do), _p(q), _p(k), _p(v), _p(tens(o)), _p(tens(lse)), _p(ev), _p(tens(dq)),
                                    _p(tens(dk)), _p(tens(dv)), B, T, Hq, Hkv, D, scale, _p(tens(wb)), nb, _stream())
    else:
        st = lib.kvs_evict_attn_varlen_fwd(_p(q), _p(k), _p(v), _p(ev), _p(cu), _p(tens(o)), _p(tens(lse)), B, ntok,
                                           mx, Hq, Hkv, D, scale, _p(tens(wf)), nf, _stream())
        assert st == 0, kvs.lib.kvs_last_error()
        st = lib.kvs_evict_attn_varlen_bwd(_p(do), _p(q), _p(k), _p(v), _p(tens(o)), _p(tens(lse)), _p(ev), _p(cu),
                                           _p(tens(dq)), _p(tens(dk)), _p(tens(dv)), B, ntok, mx, Hq, Hkv, D, scale,
                                           _p(tens(wb)), nb, _stream())
    assert st == 0, kvs.lib.kvs_last_error()
    torch.cuda.synchronize()
    outs = {name: tens(x).clone() for name, x in (("O", o), ("LSE", lse), ("dQ", dq), ("dK", dk), ("dV", dv))}
    guards = {}
    if banded:
        guards = {name: x.guards_intact() for name, x in
                  (("O", o), ("LSE", lse), ("dQ", dq), ("dK", dk), ("dV", dv), ("fwd workspace", wf),
                   ("bwd workspace", wb))}
    return outs, guards


CASES = [
    # (name, lengths, varlen, Hq, Hkv, D, layout (p, w, s), strategy)
    ("fixed B=2 L=700", [700, 700], False, 8, 2, 128, (40, 96, 24), "last2"),
    ("varlen ragged G=5", [1, 63, 640, 129, 257], True, 10, 2, 128, (17, 50, 9), "keep_all"),
    ("fixed D=64 L=333", [333], False, 6, 3, 64, (11, 40, 7), "latest_only"),
    ("split key blocks L=8704", [8704], False, 2, 1, 64, (4096, 512, 64), "keep_all"),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0].replace(" ", "_") for c in CASES])
def test_guard_bands_and_placement(kvs, case):
    name, lengths, varlen, Hq, Hkv, D, (p, w, s), strategy = case
    announce(f"canary {name}: lengths={lengths} Hq={Hq} Hkv={Hkv} D={D} varlen={varlen}")
    dev = torch.device("cuda:0")
    ntok = int(sum(lengths))
    e = np.concatenate([inputs.evict_at_layout(L, p, w, s, strategy) for L in lengths]).astype(np.int32)
    q, k, v, do = (inputs.randn_bf16(sh, 700 + i).to(dev) for i, sh in
                   enumerate([(ntok, Hq, D), (ntok, Hkv, D), (ntok, Hkv, D), (ntok, Hq, D)]))
    ev = torch.from_numpy(e).to(dev)
    scale = 1.0 / math.sqrt(D)
    if varlen:
        cu = torch.from_numpy(np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)).to(dev)
        B, T = len(lengths), None
    else:
        cu, B, T = None, len(lengths), lengths[0]
        q, k, v, do = (x.view(B, T, x.shape[1], D) for x in (q, k, v, do))
        ev = ev.view(B, T)
    plain, _ = _run(kvs, q, k, v, do, ev, cu, B, T, ntok, Hq, Hkv, D, scale, banded=False)
    banded, guards = _run(kvs, q, k, v, do, ev, cu, B, T, ntok, Hq, Hkv, D, scale, banded=True)
    bad = [g for g, ok in guards.items() if not ok]
    assert not bad, f"{name}: writes outside the buffers of {bad}"
    for key in plain:
        assert torch.equal(plain[key].view(torch.uint8), banded[key].view(torch.uint8)), \
            f"{name}: {key} differs between plain and banded buffers"


def test_paged_decode_guard_bands(kvs):
    """Decode over a small streamed cache (one sequence empty): O and LSE banded."""
    from paper_2609_35750_amd import paged

    announce("canary paged decode: S=3 bs=16 Hq=8 Hkv=2 D=128")
    dev = torch.device("cuda:0")
    S, bs, Hq, Hkv, D = 3, 16, 8, 2, 128
    cache = paged.PagedKVCache(64, bs, S, 24, Hkv, D, device=dev)
    lens = [300, 17, 0]
    for sq, L in enumerate(lens):
        if L:
            kn = inputs.randn_bf16((L, Hkv, D), 800 + sq).to(dev)
            vn = inputs.randn_bf16((L, Hkv, D), 810 + sq).to(dev)
            cache.append(sq, np.arange(L), kn, vn)
    cache.evict(0, np.arange(40, 200))
    q = inputs.randn_bf16((S, Hq, D), 820).to(dev)
    o_plain, lse_plain = cache.decode(q, 0.1)
    ob, lb = Banded((S, Hq, D), torch.bfloat16, dev), Banded((S, Hq), torch.float32, dev)
    o_b, lse_b = cache.decode(q, 0.1, out=ob.t, lse=lb.t)
    torch.cuda.synchronize()
    assert ob.guards_intact() and lb.guards_intact(), "decode wrote outside O or LSE"
    assert torch.equal(o_plain.view(torch.int16), o_b.view(torch.int16))
    assert torch.equal(lse_plain, lse_b)
