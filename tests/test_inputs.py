"""Layout rules of the synthetic traces (no GPU)."""
import numpy as np
import pytest

from oracle import attention as orc
from paper_2609_35750_amd import inputs


def test_tiny_trace_layout_spans():
    e = inputs.evict_at_layout(512, 64, 128, 32, "keep_all")
    assert (e[:64] == 512).all()
    assert (e[64:192] == 224).all() and (e[192:224] == 512).all()
    assert (e[224:352] == 384).all() and (e[352:384] == 512).all()
    assert (e[384:] == 512).all()


def test_latest_only_and_last2_summaries():
    L, p, w, s = 100, 4, 10, 2   # a = 4, 16, 28, 40, 52, 64, 76, 88, 100
    e1 = inputs.evict_at_layout(L, p, w, s, "latest_only")
    assert (e1[4:14] == 16).all()           # turns of segment 0 dropped at a_1
    assert (e1[14:16] == 28).all()          # S_0 dropped when S_1 completes (a_2)
    e2 = inputs.evict_at_layout(L, p, w, s, "last2")
    assert (e2[14:16] == 40).all()          # S_0 dropped when S_2 completes (a_3)
    # last summary of the trace: S_7 = [98, 100) completes at 100 = L -> never matters
    assert (e1[98:100] == 100).all() and (e2[98:100] == 100).all()


def test_empty_trace_in_a_varlen_batch():
    wl = inputs.custom_workload("e", 4, 2, 64, [0, 9, 0], 2, 3, 1, "last2", varlen=True)
    assert wl.ntok == 9 and list(wl.cu_seqlens()) == [0, 0, 9, 9]
    np.testing.assert_array_equal(wl.evict_at(), inputs.evict_at_layout(9, 2, 3, 1, "last2"))
    assert inputs.evict_at_layout(0, 2, 3, 1).shape == (0,)


def test_workload_sizes():
    W = inputs.WORKLOADS
    assert W["trace16k_gqa4"].ntok == 16384 and W["trace16k_gqa4"].G == 4
    assert W["trace64k_last2"].G == 8
    v = W["varlen8_gqa5"]
    assert v.B == 8 and v.G == 5 and all(4096 <= L <= 24576 for L in v.lengths)
    assert v.lengths == (24115, 14371, 8842, 15142, 19826, 6878, 10336, 10371)


@pytest.mark.parametrize("name,pairs", [("trace16k_gqa4", 58728448), ("trace32k_latest", 91766784),
                                        ("varlen8_gqa5", 251210050), ("trace64k_last2", 235372544)])
def test_visible_pairs_of_workloads(name, pairs):
    # counts derived independently when the workloads were specified
    wl = inputs.WORKLOADS[name]
    e = wl.evict_at()
    tot, off = 0, 0
    for L in wl.lengths:
        tot += int((np.minimum(e[off:off + L].astype(np.int64), L) - np.arange(L)).sum())
        off += L
    assert tot == pairs


def test_tensors_are_seeded_and_bf16():
    wl = inputs.custom_workload("t", 4, 2, 16, [33, 7], 2, 5, 1, seed=7)
    a = inputs.make_tensors(wl)
    b = inputs.make_tensors(wl)
    for key in ("q", "k", "v", "do"):
        assert str(a[key].dtype) == "torch.bfloat16"
        assert (a[key].view(-1).view(dtype=__import__("torch").int16) == b[key].view(-1).view(dtype=__import__("torch").int16)).all()
    assert a["q"].shape == (40, 4, 16) and a["k"].shape == (40, 2, 16)


# ---------------------------------------------------------------- re-prefill baseline traces
def test_reprefill_tiny_hand_count():
    # 512 tokens, p=64, w=128, s=32, keep-all: compactions 0 and 1 fire (a_1 = 224, a_2 = 384 <= 512).
    # trace 0 = [0, 224); trace 1 = prompt 64 + S_0 (32) + [224, 384); trace 2 = prompt + S_0 + S_1 + [384, 512)
    tr = inputs.reprefill_traces(512, 64, 128, 32, "keep_all")
    assert [len(t) for t in tr] == [224, 256, 256]
    assert np.array_equal(tr[1][:96], np.concatenate([np.arange(64), np.arange(192, 224)]))
    assert np.array_equal(tr[2][:128], np.concatenate([np.arange(64), np.arange(192, 224), np.arange(352, 384)]))
    ex = inputs.reprefill_extra_tokens(512, 64, 128, 32, "keep_all")
    assert ex["extra_exact"] == 224 and ex["tokens"] == 736


@pytest.mark.parametrize("strategy", inputs.STRATEGIES)
@pytest.mark.parametrize("L,p,w,s", [(60, 5, 11, 3), (97, 0, 9, 4), (40, 40, 5, 2), (88, 7, 10, 0), (50, 3, 6, 5)])
def test_reprefill_matches_stream_replay(strategy, L, p, w, s):
    """Each re-prefill trace starts with exactly the entries the streamed cache
    holds right after the compaction that opened it, and the new parts of the
    traces enumerate the rollout once."""
    import torch
    from oracle import stream_sim

    q = torch.zeros(L, 1, 4, dtype=torch.float64)
    kv = torch.zeros(L, 1, 4, dtype=torch.float64)
    _, _, lives = stream_sim.replay(q, kv, kv, p, w, s, strategy, 1.0, return_live=True)
    tr = inputs.reprefill_traces(L, p, w, s, strategy)
    pos = 0   # first token not generated yet
    for k, t in enumerate(tr):
        start = int(np.sum(t < pos))   # re-prefilled entries come first, all generated earlier
        assert np.all(t[:start] < pos) and np.array_equal(t[start:], np.arange(pos, pos + len(t) - start))
        if k == 0:
            assert start == 0
        else:
            live = [int(j) for j in lives[pos] if j != pos]   # cache right after the compaction, before token pos
            assert list(t[:start]) == live, (k, list(t[:start]), live)
        pos += len(t) - start
    assert pos == L


@pytest.mark.parametrize("strategy", inputs.STRATEGIES)
@pytest.mark.parametrize("L,p,w,s", [(512, 64, 128, 32), (60, 5, 11, 3), (97, 0, 9, 4), (88, 7, 10, 0), (16384, 1024, 4096, 512)])
def test_reprefill_from_evict_matches_layout_builder(strategy, L, p, w, s):
    """Deriving the fresh traces from evict_at alone gives the segment builder's traces."""
    a = inputs.reprefill_traces(L, p, w, s, strategy)
    b = inputs.reprefill_traces_from_evict(inputs.evict_at_layout(L, p, w, s, strategy))
    assert len(a) == len(b) and all(np.array_equal(x, y) for x, y in zip(a, b))


@pytest.mark.parametrize("strategy,window,stride,keep", [("sliding_window", 4, 1, 0), ("markovian_thinker", 6, 0, 0),
                                                         ("markovian_pick", 5, 0, 2)])
def test_reprefill_from_evict_turns_match_replay(strategy, window, stride, keep):
    from oracle import stream_sim

    rng = np.random.default_rng(5)
    lengths = inputs.turn_lengths(15, 1, 6, rng)
    picks = inputs.pick_turns(15, window, keep, rng) if strategy == "markovian_pick" else None
    e = inputs.evict_at_turns(4, lengths, strategy, window, stride=stride, picks=picks)
    lives = stream_sim.live_sets_turns(4, lengths, strategy, window, stride=stride, picks=picks)
    pos = 0
    for k, t in enumerate(inputs.reprefill_traces_from_evict(e)):
        start = int(np.sum(t < pos))
        if k:
            assert list(t[:start]) == [int(j) for j in lives[pos] if j != pos]
        pos += len(t) - start
    assert pos == len(e)
