"""Streamed paged KV cache, CPU tier: pins of the decode oracle and the host
block manager of libkvs (no GPU needed; the block manager makes no HIP call).

Decode (Section 2, "KV-streams"): the query generated at trace position t
attends over the cache entries live at that moment, R(t) = {j <= t: e_j > t};
that is row t of the eviction-masked attention.
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import attention as orc
from oracle import paged as opg
from oracle import stream_sim
from paper_2609_35750_amd import inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_35750_amd", "libkvs.so")


# ---------------------------------------------------------------- oracle pins
@pytest.mark.parametrize("strategy", inputs.STRATEGIES)
def test_live_set_matches_stream_replay(strategy):
    """The live set from the eviction indices equals the cache the stream replay
    builds from the strategy description alone."""
    L, p, w, s = 150, 9, 17, 5
    e = inputs.evict_at_layout(L, p, w, s, strategy)
    q, k, v = (inputs.randn_bf16(sh, 7 + i) for i, sh in enumerate([(L, 2, 8), (L, 1, 8), (L, 1, 8)]))
    _, _, lives = stream_sim.replay(q.double(), k.double(), v.double(), p, w, s, strategy, 0.3, return_live=True)
    for t in range(L):
        np.testing.assert_array_equal(opg.live_set(e, t), np.sort(lives[t]))


def test_turn_live_sets_match_replay():
    rng = np.random.default_rng(3)
    lengths = inputs.turn_lengths(14, 1, 9, rng, pad=4)
    e = inputs.evict_at_turns(6, lengths, "sliding_window", 4, stride=1)
    lives = stream_sim.live_sets_turns(6, lengths, "sliding_window", 4, stride=1)
    for t in range(len(e)):
        np.testing.assert_array_equal(opg.live_set(e, t), np.sort(lives[t]))


@pytest.mark.parametrize("strategy", inputs.STRATEGIES)
def test_decode_equals_masked_attention_rows(strategy):
    """Decoding every token over its live set reproduces the masked forward (O, LSE)."""
    L, Hq, Hkv, D = 120, 6, 2, 16
    e = inputs.evict_at_layout(L, 8, 20, 6, strategy)
    q, k, v = (inputs.randn_bf16(sh, 20 + i) for i, sh in enumerate([(L, Hq, D), (L, Hkv, D), (L, Hkv, D)]))
    scale = 1.0 / math.sqrt(D)
    O, LSE = orc.forward(q, k, v, e, scale)
    for t in range(L):
        o, lse = opg.decode(q[t], k, v, opg.live_set(e, t), scale)
        np.testing.assert_allclose(o, O[t], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse, LSE[:, t], rtol=1e-12, atol=1e-12)


def test_decode_closed_forms():
    rng = np.random.default_rng(1)
    q, k, v = rng.standard_normal((4, 8)), rng.standard_normal((10, 2, 8)), rng.standard_normal((10, 2, 8))
    # one live entry: O = v_j, LSE = s_j
    o, lse = opg.decode(q, k, v, [6], 0.5)
    np.testing.assert_allclose(o, v[6, [0, 0, 1, 1]], rtol=0, atol=1e-15)
    np.testing.assert_allclose(lse, 0.5 * np.einsum("hd,hd->h", q, k[6, [0, 0, 1, 1]]), rtol=1e-13, atol=1e-15)
    # the order of the cache entries does not matter; duplicates of equal scores shift LSE by ln 2
    a = opg.decode(q, k, v, [1, 4, 7, 9], 0.5)
    b = opg.decode(q, k, v, [9, 1, 7, 4], 0.5)
    np.testing.assert_allclose(a[0], b[0], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(a[1], b[1], rtol=1e-13, atol=1e-14)
    o2, lse2 = opg.decode(q, k, v, [3, 3], 0.5)
    o1, lse1 = opg.decode(q, k, v, [3], 0.5)
    np.testing.assert_allclose(o2, o1, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(lse2, lse1 + math.log(2), rtol=1e-14)
    # empty cache
    o, lse = opg.decode(q, k, v, [], 0.5)
    assert np.all(o == 0) and np.all(np.isneginf(lse))
    # uniform scores: O is the plain mean of the live values
    o, _ = opg.decode(np.zeros((4, 8)), k, v, [0, 2, 5], 1.0)
    np.testing.assert_allclose(o[0], v[[0, 2, 5], 0].mean(axis=0), rtol=1e-14)


# ---------------------------------------------------------------- host block manager
needs_lib = pytest.mark.skipif(not os.path.exists(LIB), reason="libkvs.so not built (run __graft_entry__.build())")


def _bm(*args):
    from paper_2609_35750_amd.paged import BlockManager

    return BlockManager(*args)


def _replay_events(e):
    """Per time t: positions to evict (e_j == t) before token t is appended."""
    L = len(e)
    ev = [[] for _ in range(L)]
    for j, x in enumerate(np.minimum(e, L)):
        if x < L:
            ev[x].append(j)
    return ev


@needs_lib
@pytest.mark.parametrize("bs", [1, 16, 5])
def test_block_manager_tracks_live_sets(bs):
    """Three sequences with different strategies share one pool: after every
    step the cached positions of each sequence are exactly R(t), slots are
    unique and lie in the sequence's own listed blocks, and every block is
    either free or used by exactly one sequence."""
    L = 260
    es = [inputs.evict_at_layout(L, 10, 40, 8, st) for st in inputs.STRATEGIES]
    nb = 3 * (L // bs + 4)
    bm = _bm(nb, bs, 3, L // bs + 4)
    slot_of = [dict() for _ in es]
    evs = [_replay_events(e) for e in es]
    for t in range(L):
        for s, e in enumerate(es):
            if evs[s][t]:
                slots = bm.evict(s, evs[s][t])
                for j, sl in zip(evs[s][t], slots):
                    assert slot_of[s].pop(j) == sl
            sl = bm.append(s, [t])
            slot_of[s][t] = int(sl[0])
        if t % 13 == 0 or t == L - 1:
            table, nblk = bm.tables()
            owner = {}
            for s, e in enumerate(es):
                assert sorted(slot_of[s]) == list(opg.live_set(e, t))
                assert bm.live(s) == len(slot_of[s])
                blocks = list(table[s, : nblk[s]])
                for b in blocks:
                    assert b not in owner
                    owner[b] = s
                for sl in slot_of[s].values():
                    assert sl // bs in blocks
                # every listed block still holds a live entry of its sequence
                assert {sl // bs for sl in slot_of[s].values()} == set(blocks)
            assert len(owner) + bm.free_blocks() == nb
            allslots = [sl for d in slot_of for sl in d.values()]
            assert len(allslots) == len(set(allslots))


@needs_lib
def test_block_manager_reuses_freed_blocks_and_releases():
    bm = _bm(4, 4, 2, 4)
    a = bm.append(0, range(8))                      # blocks 0, 1
    assert list(a) == list(range(8)) and bm.free_blocks() == 2
    bm.evict(0, [0, 1, 2])                          # block 0 still has position 3
    assert bm.free_blocks() == 2
    bm.evict(0, [3])                                # block 0 free again
    assert bm.free_blocks() == 3
    b = bm.append(1, range(4))                      # takes the freed block 0 first (LIFO)
    assert sorted(b // 4) == [0, 0, 0, 0]
    table, nblk = bm.tables()
    assert list(table[0, : nblk[0]]) == [1] and list(table[1, : nblk[1]]) == [0]
    # evicting the tail block of a sequence makes the next append open a new block
    bm.evict(0, [4, 5, 6, 7])
    assert bm.live(0) == 0 and bm.free_blocks() == 3
    c = bm.append(0, [100])
    assert bm.free_blocks() == 2 and c[0] % 4 == 0
    rel = bm.release(1)
    assert sorted(rel) == sorted(b) and bm.free_blocks() == 3 and bm.live(1) == 0


@needs_lib
def test_block_manager_errors_are_all_or_nothing():
    from paper_2609_35750_amd.kvs import KVS_ERR_CAPACITY, KVS_ERR_SHAPE, KVS_ERR_STATE, KvsError

    bm = _bm(2, 4, 2, 8)
    bm.append(0, range(6))
    with pytest.raises(KvsError) as ex:
        bm.append(1, range(5))                      # needs 2 blocks, 0 free
    assert ex.value.status == KVS_ERR_CAPACITY and bm.live(1) == 0 and bm.free_blocks() == 0
    with pytest.raises(KvsError) as ex:
        bm.append(0, [6, 7, 5])                     # 5 already cached
    assert ex.value.status == KVS_ERR_STATE and bm.live(0) == 6
    with pytest.raises(KvsError) as ex:
        bm.append(0, [6, 6])
    assert ex.value.status == KVS_ERR_STATE
    with pytest.raises(KvsError) as ex:
        bm.evict(0, [1, 99])                        # 99 not cached: nothing evicted
    assert ex.value.status == KVS_ERR_STATE and bm.live(0) == 6
    with pytest.raises(KvsError) as ex:
        bm.evict(0, [2, 2])
    assert ex.value.status == KVS_ERR_STATE and bm.live(0) == 6
    with pytest.raises(KvsError) as ex:
        bm.append(2, [0])
    assert ex.value.status == KVS_ERR_SHAPE
    small = _bm(8, 2, 1, 2)                         # table of 2 blocks per sequence
    small.append(0, range(4))
    with pytest.raises(KvsError) as ex:
        small.append(0, [4])
    assert ex.value.status == KVS_ERR_CAPACITY


@needs_lib
def test_paged_abi_validation():
    from paper_2609_35750_amd import kvs as k

    L, FAKE = k.lib, 1 << 20
    with pytest.raises(k.KvsError):
        _bm(0, 16, 1, 1)
    with pytest.raises(k.KvsError):
        _bm(4, 65, 1, 1)
    need = L.kvs_paged_decode_workspace(2, 8, 2, 128, 16, 16)
    assert need > 0

    def dec(S=2, Hq=8, Hkv=2, D=128, nb=64, bs=16, mb=16, scale=0.1, ws=FAKE, nbytes=None, q=FAKE):
        return L.kvs_paged_decode(q, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, S, Hq, Hkv, D, nb, bs, mb, scale,
                                  ws, need if nbytes is None else nbytes, None)

    assert dec(D=96) == k.KVS_ERR_SHAPE
    assert dec(Hq=6, Hkv=4) == k.KVS_ERR_SHAPE
    assert dec(bs=65) == k.KVS_ERR_SHAPE
    assert dec(Hq=66, Hkv=1) == k.KVS_ERR_UNSUPPORTED
    assert dec(q=None) == k.KVS_ERR_NULL
    assert dec(q=FAKE + 4) == k.KVS_ERR_ALIGN
    assert dec(nbytes=need - 1) == k.KVS_ERR_WORKSPACE
    assert dec(scale=-1.0) == k.KVS_ERR_SHAPE
    assert L.kvs_paged_append(FAKE, FAKE, FAKE, FAKE, 4, FAKE, FAKE, FAKE, 8, 16, 2, 80, None) == k.KVS_ERR_SHAPE
    assert L.kvs_paged_append(FAKE, FAKE, None, FAKE, 4, FAKE, FAKE, FAKE, 8, 16, 2, 64, None) == k.KVS_ERR_NULL
    assert L.kvs_paged_evict(FAKE, -1, FAKE, 8, 16, None) == k.KVS_ERR_SHAPE
    assert L.kvs_paged_evict(None, 3, FAKE, 8, 16, None) == k.KVS_ERR_NULL


@needs_lib
@pytest.mark.parametrize("seed", range(4))
def test_block_manager_random_operations_match_model(seed):
    """Random appends, evictions and releases over several sequences against a
    plain model of the rules (tokens fill the tail of the last block, evicted
    slots are never refilled, a block is freed when none of its entries is
    live): live sets, per-sequence block counts and the free-block count agree
    after every operation, and failed operations change nothing."""
    from paper_2609_35750_amd.kvs import KvsError

    rng = np.random.default_rng(seed)
    nb, bs, S, mb = int(rng.integers(6, 20)), int(rng.choice([1, 2, 4, 16])), 3, 8
    bm = _bm(nb, bs, S, mb)
    live = [dict() for _ in range(S)]          # position -> slot
    nxt = [0] * S
    for _ in range(400):
        s = int(rng.integers(0, S))
        op = rng.random()
        try:
            if op < 0.55:
                n = int(rng.integers(1, 2 * bs + 2))
                pos = list(range(nxt[s], nxt[s] + n))
                slots = bm.append(s, pos)
                nxt[s] += n
                live[s].update(zip(pos, (int(x) for x in slots)))
            elif op < 0.9 and live[s]:
                k = int(rng.integers(1, len(live[s]) + 1))
                pos = [int(x) for x in rng.choice(sorted(live[s]), size=k, replace=False)]
                slots = bm.evict(s, pos)
                for p_, sl in zip(pos, slots):
                    assert live[s].pop(p_) == sl
            elif op >= 0.9:
                rel = bm.release(s)
                assert sorted(rel) == sorted(live[s].values())
                live[s].clear()
        except KvsError:
            pass                                # capacity: the model keeps its state too
        table, nblk = bm.tables()
        used = set()
        for q in range(S):
            assert bm.live(q) == len(live[q])
            blocks = set(int(b) for b in table[q, : nblk[q]])
            # every live slot lies in a listed block; every listed block but the tail holds a live entry
            assert {sl // bs for sl in live[q].values()} <= blocks
            assert len(blocks - {sl // bs for sl in live[q].values()}) <= 1
            assert not (blocks & used)
            used |= blocks
        assert len(used) + bm.free_blocks() == nb
        allslots = [sl for d in live for sl in d.values()]
        assert len(allslots) == len(set(allslots))
