"""Streamed paged KV cache on the GPU vs the fp64 oracle (MI355X).

A rollout is replayed token by token the way the inference engine runs it
(Section 2, "KV-streams"; Section 4, "Inference engine implementation"):
before token t is generated, the entries whose eviction index is t are
dropped from the cache (kvs_bm_evict + kvs_paged_evict), then token t's K and
V are appended (kvs_bm_append + kvs_paged_append).  At sampled steps every
sequence decodes its query q_t over its live cache (kvs_paged_decode), which
must equal the oracle's attention over R(t) = {j <= t : e_j > t}, i.e. row t
of the eviction-masked attention the trainer computes.  Several sequences with
different strategies share one block pool, so freed blocks are reused across
sequences.  Every case prints its name before it runs.
"""
import math

import numpy as np
import pytest
import torch

from oracle import paged as opg
from paper_2609_35750_amd import inputs
from tests.gpu_helpers import REL_L2, announce, assert_close, assert_flat, assert_lse, to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pg():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35750_amd import paged

    return paged


def _events(e, L):
    ev = [[] for _ in range(L)]
    for j, x in enumerate(np.minimum(np.asarray(e, dtype=np.int64), L)):
        if x < L:
            ev[x].append(j)
    return ev


def _stream(pg, seqs, bs, Hkv, D, samples, nb=None, max_blocks=None, scale=None):
    """Replay the sequences (dicts with e, q, k, v on the CPU) through one cache;
    returns {t: (O [S,Hq,D], LSE [S,Hq])} at the sampled steps, and the cache."""
    dev = torch.device("cuda:0")
    S = len(seqs)
    Lmax = max(len(s["e"]) for s in seqs)
    max_blocks = max_blocks or (Lmax + bs - 1) // bs + 2
    nb = nb or S * max_blocks
    cache = pg.PagedKVCache(nb, bs, S, max_blocks, Hkv, D, device=dev)
    evs = [_events(s["e"], len(s["e"])) for s in seqs]
    kd = [s["k"].to(dev) for s in seqs]
    vd = [s["v"].to(dev) for s in seqs]
    Hq = seqs[0]["q"].shape[1]
    scale = scale or 1.0 / math.sqrt(D)
    out = {}
    for t in range(Lmax):
        for i, s in enumerate(seqs):
            if t >= len(s["e"]):
                continue
            if evs[i][t]:
                cache.evict(i, evs[i][t])
            cache.append(i, [t], kd[i][t:t + 1], vd[i][t:t + 1])
        if t in samples:
            q = torch.stack([s["q"][min(t, len(s["e"]) - 1)] for s in seqs]).to(dev)
            o, lse = cache.decode(q, scale)
            torch.cuda.synchronize()
            out[t] = (o.cpu(), lse.cpu())
    return out, cache


def _check(name, seqs, out, scale):
    for t, (o, lse) in out.items():
        for i, s in enumerate(seqs):
            if t >= len(s["e"]):
                continue
            ro, rl = opg.decode(s["q"][t], s["k"], s["v"], opg.live_set(s["e"], t), scale)
            assert_close(f"{name} t={t} seq={i} O", to_f64(o[i]), ro)
            assert_lse(f"{name} t={t} seq={i}", to_f64(lse[i]), rl)


def _seq(e, Hq, Hkv, D, seed):
    L = len(e)
    q, k, v = (inputs.randn_bf16(sh, seed + i) for i, sh in enumerate([(L, Hq, D), (L, Hkv, D), (L, Hkv, D)]))
    return {"e": np.asarray(e, dtype=np.int64), "q": q, "k": k, "v": v}


def _samples(L, e):
    """First token, each eviction time and the step after it, a few random steps, the last token."""
    ts = {0, L - 1}
    for x in np.unique(np.minimum(e, L)):
        if x < L:
            ts.update({int(x), min(int(x) + 1, L - 1)})
    rng = np.random.default_rng(L)
    ts.update(int(x) for x in rng.integers(0, L, 4))
    return sorted(ts)


CASES = [
    # (block size, Hq, Hkv, D, L, p, w, s)
    (16, 8, 2, 128, 700, 40, 96, 24),
    (1, 4, 4, 64, 420, 17, 50, 9),
    (16, 16, 2, 128, 520, 32, 64, 16),
    (5, 6, 3, 64, 333, 11, 40, 7),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"bs{c[0]}_H{c[1]}x{c[2]}_D{c[3]}_L{c[4]}")
def test_decode_over_streamed_cache_matches_masked_rows(pg, case):
    bs, Hq, Hkv, D, L, p, w, s = case
    announce(f"paged stream bs={bs} Hq={Hq} Hkv={Hkv} D={D} L={L} layout=({p},{w},{s}) x 3 strategies")
    seqs = [_seq(inputs.evict_at_layout(L, p, w, s, st), Hq, Hkv, D, 40 + 5 * i)
            for i, st in enumerate(inputs.STRATEGIES)]
    samples = set()
    for sq in seqs:
        samples.update(_samples(L, sq["e"]))
    out, cache = _stream(pg, seqs, bs, Hkv, D, samples)
    _check(f"bs{bs}", seqs, out, 1.0 / math.sqrt(D))
    # cache contents: live slots hold exactly R(L-1), with the appended K/V bits
    slot_pos = cache.slot_pos.cpu().numpy()
    table, nblk = cache.bm.tables()
    # [block][Hkv][row][D] -> per slot [slot][Hkv][D]
    kc = cache.k.cpu().view(torch.int16).numpy().transpose(0, 2, 1, 3).reshape(-1, Hkv, D)
    for i, sq in enumerate(seqs):
        slots = np.concatenate([np.arange(b * bs, (b + 1) * bs) for b in table[i, : nblk[i]]]) if nblk[i] else []
        pos = slot_pos[slots]
        live = np.sort(pos[pos >= 0])
        np.testing.assert_array_equal(live, opg.live_set(sq["e"], L - 1))
        sl = np.asarray(slots)[pos >= 0]
        np.testing.assert_array_equal(kc[sl], sq["k"].view(torch.int16).numpy()[pos[pos >= 0]])


def test_turn_level_sliding_window_padded_blocks(pg):
    """Turns padded to 16 tokens (the vLLM setup): evictions free whole blocks."""
    rng = np.random.default_rng(9)
    lengths = inputs.turn_lengths(24, 8, 40, rng, pad=16)
    e = inputs.evict_at_turns(32, lengths, "sliding_window", 5, stride=1)
    L = len(e)
    announce(f"paged sliding window bs=16 L={L} G=8")
    seqs = [_seq(e, 16, 2, 128, 70), _seq(inputs.evict_at_turns(32, lengths, "markovian_thinker", 6), 16, 2, 128, 80)]
    out, cache = _stream(pg, seqs, 16, 2, 128, set(_samples(L, e)))
    _check("turns", seqs, out, 1.0 / math.sqrt(128))


def test_empty_and_single_entry_sequences(pg):
    dev = torch.device("cuda:0")
    announce("paged empty / single-entry sequences")
    cache = pg.PagedKVCache(8, 16, 3, 4, 2, 128, device=dev)
    k1, v1 = inputs.randn_bf16((1, 2, 128), 1), inputs.randn_bf16((1, 2, 128), 2)
    cache.append(1, [0], k1.to(dev), v1.to(dev))
    k2, v2 = inputs.randn_bf16((3, 2, 128), 3), inputs.randn_bf16((3, 2, 128), 4)
    cache.append(2, [0, 1, 2], k2.to(dev), v2.to(dev))
    cache.evict(2, [0, 1, 2])          # block freed again: nothing live
    q = inputs.randn_bf16((3, 4, 128), 5)
    o, lse = cache.decode(q.to(dev), 0.1)
    o, lse = to_f64(o), to_f64(lse)
    assert np.all(o[0] == 0) and np.all(np.isneginf(lse[0]))
    assert np.all(o[2] == 0) and np.all(np.isneginf(lse[2]))
    ro, rl = opg.decode(q[1], k1, v1, [0], 0.1)
    assert_flat("single O", o[1], ro, 4e-3, REL_L2)          # one entry: O = v (bf16-exact up to rounding)
    assert_lse("single", lse[1], rl)


def test_long_cache_many_splits(pg):
    """A long keep-all trace decoded by two sequences: the key range is cut
    into many splits (several empty for the shorter sequence) and merged."""
    L = 9000
    announce(f"paged long cache L={L} bs=16 G=4")
    e = inputs.evict_at_layout(L, 1024, 2048, 256, "keep_all")
    seqs = [_seq(e, 8, 2, 128, 90), _seq(inputs.evict_at_layout(3000, 100, 500, 50, "latest_only"), 8, 2, 128, 95)]
    out, _ = _stream(pg, seqs, 16, 2, 128, {2999, 4500, L - 1})
    _check("long", seqs, out, 1.0 / math.sqrt(128))


def test_bench_configuration_sampled(pg):
    """The decode bench.py times: 64 rollouts of the 16k keep-all trace
    (Hq=32, Hkv=8, D=128) streamed segment by segment through one 16-token
    block cache, decoded at token 16,383.  Rollouts 0, 31 and 63 carry seeded
    CPU inputs and are compared with the oracle over R(L-1); the others get
    seeded GPU noise of the same shape (they share and reuse the block pool)."""
    dev = torch.device("cuda:0")
    S, L, p, w, s_, Hq, Hkv, D, bs = 64, 16384, 1024, 4096, 512, 32, 8, 128, 16
    announce(f"paged bench configuration S={S} L={L} Hq={Hq} Hkv={Hkv} D={D} bs={bs}")
    e = inputs.evict_at_layout(L, p, w, s_, "keep_all")
    live = opg.live_set(e, L - 1)
    max_blocks = (L + bs - 1) // bs + 1
    nb = S * ((len(live) + w + s_) // bs + 4)
    cache = pg.PagedKVCache(nb, bs, S, max_blocks, Hkv, D, device=dev)
    checked = {0: 900, 31: 910, 63: 920}
    gen = torch.Generator(device=dev)
    gen.manual_seed(77)
    ev_t = {}
    for j, x in enumerate(np.minimum(e, L)):
        if x < L:
            ev_t.setdefault(int(x), []).append(j)
    cuts = sorted(set(ev_t) | {L})
    kv = {}
    for sq in range(S):
        if sq in checked:
            kv[sq] = (inputs.randn_bf16((L, Hkv, D), checked[sq]), inputs.randn_bf16((L, Hkv, D), checked[sq] + 1))
        t0 = 0
        for t1 in cuts:
            if t0 < t1:
                if sq in checked:
                    kn, vn = kv[sq][0][t0:t1].to(dev), kv[sq][1][t0:t1].to(dev)
                else:
                    kn = torch.randn((t1 - t0, Hkv, D), generator=gen, device=dev).to(torch.bfloat16)
                    vn = torch.randn((t1 - t0, Hkv, D), generator=gen, device=dev).to(torch.bfloat16)
                cache.append(sq, np.arange(t0, t1), kn, vn)
            if t1 < L:
                cache.evict(sq, ev_t[t1])
            t0 = t1
    q = inputs.randn_bf16((S, Hq, D), 930)
    o, lse = cache.decode(q.to(dev), 1.0 / math.sqrt(D))
    o, lse = to_f64(o), to_f64(lse)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    for sq in checked:
        ro, rl = opg.decode(q[sq], kv[sq][0], kv[sq][1], live, 1.0 / math.sqrt(D))
        assert_close(f"bench-config seq={sq} O", o[sq], ro)
        assert_lse(f"bench-config seq={sq}", lse[sq], rl)
