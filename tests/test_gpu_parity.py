"""HIP path vs the fp64 oracle, element by element, on seeded inputs (MI355X).

Sizes here are ones the oracle finishes in seconds while still spanning
several tiles and ragged tails.  Every case prints its name before it runs.
"""
import numpy as np
import pytest
import torch

from oracle import attention as orc
from oracle import tiles as otiles
from paper_2609_35750_amd import inputs
from tests.gpu_helpers import (announce, assert_close, assert_flat, assert_lse, assert_switches_bitwise,
                               gpu_fwd_bwd, to_f64)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kvs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35750_amd import kvs as k

    return k


def _parity(kvs, wl, e, cu=None, B=None, switches=True, q_mul=None, max_seqlen=None):
    """Element by element against the oracle; then the tile-classifier
    switches must leave every output bit-identical.  q_mul (a power of two, so
    the bf16 query stays exact) widens the logits; max_seqlen (varlen) may
    exceed the longest trace."""
    t = inputs.make_tensors(wl)
    if q_mul is not None:
        t["q"] = t["q"] * q_mul
    scale = wl.softmax_scale
    mx = (max_seqlen or max(wl.lengths)) if cu is not None else None
    announce(f"{wl.name} lengths={wl.lengths} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D} varlen={cu is not None} B={B} "
             f"max_seqlen={mx}")
    res = gpu_fwd_bwd(kvs, t["q"], t["k"], t["v"], t["do"], e, scale, cu_seqlens=cu, max_seqlen=mx, B=B)
    cu_ref = cu if cu is not None else (np.arange(B + 1) * wl.lengths[0] if B else None)
    ref = orc.backward(t["q"], t["k"], t["v"], e, scale, t["do"], cu_seqlens=cu_ref)
    E = orc.dq_rounding_scale(t["q"], t["k"], t["v"], e, scale, t["do"], np.arange(wl.ntok), cu_seqlens=cu_ref)
    SK, SV = orc.dkdv_rounding_rss(t["q"], t["k"], t["v"], e, scale, t["do"], cu_seqlens=cu_ref)
    out = {}
    for key in ("O", "dq", "dk", "dv"):
        out[key] = assert_close(f"{wl.name}:{key}", to_f64(res[key]), ref[key], E=E if key == "dq" else None,
                                S={"dk": SK, "dv": SV}.get(key))
    assert_lse(wl.name, to_f64(res["LSE"]), ref["LSE"])
    if switches:
        assert_switches_bitwise(kvs, res, t["q"], t["k"], t["v"], t["do"], e, scale, cu_seqlens=cu, max_seqlen=mx,
                                B=B, label=wl.name)
    return out


def test_tiny_trace_all_outputs(kvs):
    wl = inputs.WORKLOADS["trace512_tiny"]
    _parity(kvs, wl, wl.evict_at())


LAYOUT_CASES = [
    # (L, Hq, Hkv, D, p, w, s, strategy)
    (1, 2, 2, 64, 0, 1, 0, "keep_all"),
    (17, 4, 4, 128, 3, 5, 2, "keep_all"),
    (100, 8, 2, 128, 10, 30, 7, "latest_only"),
    (257, 5, 1, 128, 16, 48, 16, "last2"),
    (300, 8, 1, 64, 20, 64, 16, "keep_all"),
    (641, 6, 2, 128, 64, 128, 32, "last2"),
    (700, 3, 3, 64, 33, 97, 13, "latest_only"),
    (1024, 16, 2, 128, 64, 200, 40, "keep_all"),
    # no permanent prompt: the first keys are evicted, so rows of a wave that see nothing in a key
    # tile share it with rows that do (the forward's wave-wide rescale must leave them finite)
    (1000, 4, 2, 128, 0, 100, 20, "keep_all"),
    (1000, 4, 2, 64, 0, 100, 20, "latest_only"),
    (777, 8, 1, 128, 0, 60, 12, "last2"),
    (520, 6, 3, 64, 0, 37, 5, "keep_all"),
]


@pytest.mark.parametrize("case", LAYOUT_CASES, ids=lambda c: f"L{c[0]}_H{c[1]}x{c[2]}_D{c[3]}_{c[7]}")
def test_layouts(kvs, case):
    L, Hq, Hkv, D, p, w, s, strat = case
    wl = inputs.custom_workload(f"layout_L{L}", Hq, Hkv, D, [L], p, w, s, strat, seed=L)
    _parity(kvs, wl, wl.evict_at())


# Head-group shapes away from the benchmarked ones: the row kernels' head grouping
# (4, 2 or 1 q-heads per workgroup, whichever divides G), the dK/dV kernel's
# G q-heads per KV head, KV-head counts that are not a multiple of the 8 XCDs,
# and the largest group size the library accepts (64).
GROUP_CASES = [
    # (L, Hq, Hkv, D)
    (300, 32, 2, 128),   # G = 16
    (257, 12, 12, 64),   # G = 1, 12 KV heads
    (200, 64, 1, 64),    # G = 64
    (333, 24, 8, 128),   # G = 3
    (190, 14, 2, 128),   # G = 7
]


@pytest.mark.parametrize("case", GROUP_CASES, ids=lambda c: f"L{c[0]}_H{c[1]}x{c[2]}_D{c[3]}")
def test_group_shapes(kvs, case):
    L, Hq, Hkv, D = case
    wl = inputs.custom_workload(f"group_L{L}_G{Hq // Hkv}", Hq, Hkv, D, [L], 9, 41, 7, "last2", seed=L + Hq)
    _parity(kvs, wl, wl.evict_at())


@pytest.mark.parametrize("D", [128, 64])
def test_large_logits(kvs, D):
    """Scores 16 times wider than unit-variance inputs give (standard deviation
    ~16 at scale 1/sqrt(D)): nearly one-hot softmax rows, exponentials far
    below fp32 range, and a reference maximum that keeps moving by more than
    the forward's lazy-rescale margin (8 in log2 units) as the walk proceeds."""
    wl = inputs.custom_workload(f"wide_logits_D{D}", 8, 2, D, [700], 12, 60, 10, "last2", seed=700 + D)
    _parity(kvs, wl, wl.evict_at(), q_mul=16.0)


@pytest.mark.parametrize("L,Hq,Hkv,D,seed", [(130, 4, 2, 128, 1), (333, 2, 1, 64, 2), (515, 10, 2, 128, 3)])
def test_random_evict_at(kvs, L, Hq, Hkv, D, seed):
    wl = inputs.custom_workload(f"random_L{L}", Hq, Hkv, D, [L], 0, 1, 0, seed=seed + 50)
    e = inputs.evict_at_random(L, np.random.default_rng(seed))
    _parity(kvs, wl, e)


def test_fixed_batch_of_traces(kvs):
    wl = inputs.custom_workload("batch3", 4, 2, 128, [200, 200, 200], 8, 40, 8, "latest_only", varlen=False, seed=9)
    _parity(kvs, wl, wl.evict_at(), B=3)


def test_varlen_ragged(kvs):
    wl = inputs.custom_workload("varlen_small", 10, 2, 128, [37, 1, 300, 129, 64], 4, 50, 10, "keep_all",
                                varlen=True, seed=13)
    _parity(kvs, wl, wl.evict_at(), cu=wl.cu_seqlens())


@pytest.mark.parametrize("D", [128, 64])
def test_varlen_loose_max_seqlen(kvs, D):
    """max_seqlen only bounds the trace lengths: three times the longest (grids
    and the dK/dV plan sized for longer traces than there are) gives the same
    parity, including split slots sized for traces that are not there."""
    wl = inputs.custom_workload(f"varlen_loose_D{D}", 6, 2, D, [37, 1, 300, 129, 0, 64], 4, 50, 10, "latest_only",
                                varlen=True, seed=21 + D)
    _parity(kvs, wl, wl.evict_at(), cu=wl.cu_seqlens(), max_seqlen=3 * max(wl.lengths))
    wl = inputs.custom_workload(f"varlen_loose_split_D{D}", 4, 2, D, [300, 1200], 64, 200, 20, "keep_all",
                                varlen=True, seed=25 + D)
    _parity(kvs, wl, wl.evict_at(), cu=wl.cu_seqlens(), max_seqlen=9000)


def test_varlen_without_prompt(kvs):
    wl = inputs.custom_workload("varlen_p0", 8, 2, 128, [300, 1, 700, 129, 64], 0, 50, 10, "latest_only",
                                varlen=True, seed=14)
    _parity(kvs, wl, wl.evict_at(), cu=wl.cu_seqlens())


@pytest.mark.parametrize("D", [128, 64])
def test_varlen_with_empty_traces(kvs, D):
    """Empty traces inside the batch, at its start and at its end (a trace whose
    start is Ntot): every kernel skips them and the others are unaffected."""
    wl = inputs.custom_workload(f"varlen_empty_D{D}", 6, 2, D, [0, 37, 0, 300, 129, 0], 4, 50, 10, "last2",
                                varlen=True, seed=15 + D)
    _parity(kvs, wl, wl.evict_at(), cu=wl.cu_seqlens())


def test_empty_batch(kvs):
    """Ntot = 0: forward and backward return zero-size outputs and enqueue nothing."""
    dev = torch.device("cuda:0")
    announce("empty batch Ntot=0")
    q = torch.empty(0, 4, 64, dtype=torch.bfloat16, device=dev)
    k = torch.empty(0, 2, 64, dtype=torch.bfloat16, device=dev)
    ev = torch.empty(0, dtype=torch.int32, device=dev)
    cu = torch.zeros(3, dtype=torch.int32, device=dev)
    o, lse = kvs.kvs_evict_attn_fwd(q, k, k, ev, cu_seqlens=cu, max_seqlen=1)
    assert o.shape == q.shape and lse.shape == (4, 0)
    dq, dk, dv = kvs.kvs_evict_attn_bwd(q, q, k, k, o, lse, ev, cu_seqlens=cu, max_seqlen=1)
    assert dq.shape == q.shape and dk.shape == k.shape and dv.shape == k.shape
    torch.cuda.synchronize()


@pytest.mark.parametrize("D", [128, 64])
def test_turn_sliding_window_without_prompt(kvs, D):
    turns = ("sliding_window", 4, 1, 0, 20, 100, 1, 99 + D)
    wl = inputs.custom_workload(f"turns_p0_D{D}", 8, 2, D, [900], 0, 0, 0, seed=98 + D, turns=turns)
    _parity(kvs, wl, wl.evict_at())


def test_varlen_many_short_traces(kvs):
    """48 packed traces of 1-160 tokens (most shorter than one tile, many
    tile-straddling offsets): per-trace indexing, tails and tile statistics."""
    rng = np.random.default_rng(2024)
    lengths = [int(x) for x in rng.integers(1, 161, 48)]
    wl = inputs.custom_workload("varlen_many", 6, 3, 64, lengths, 9, 30, 6, "latest_only", varlen=True, seed=17)
    _parity(kvs, wl, wl.evict_at(), cu=wl.cu_seqlens())


def test_varlen_600_traces(kvs):
    """600 packed traces of 0-300 tokens: more traces than the dK/dV plan groups
    by trace (it then orders work items by length alone), trace indices in the
    hundreds in every kernel's addressing, and empty traces among them."""
    rng = np.random.default_rng(600)
    lengths = [int(x) for x in rng.integers(0, 301, 600)]
    wl = inputs.custom_workload("varlen_600", 4, 2, 128, lengths, 16, 60, 12, "last2", varlen=True, seed=600)
    assert wl.B > 256 and 0 in lengths
    _parity(kvs, wl, wl.evict_at(), cu=wl.cu_seqlens())


# Traces past 8192 rows have key blocks (the prompt) visible to more than two
# 4096-row chunks: the dK/dV work is then split into row chunks whose fp32
# partial sums are added afterwards.  Element-by-element parity and bitwise
# reproducibility of that path, fixed-length and packed.
@pytest.mark.parametrize("L,Hq,Hkv,D", [(8704, 2, 1, 64), (8385, 4, 2, 128)])
def test_long_key_spans_split(kvs, L, Hq, Hkv, D):
    wl = inputs.custom_workload(f"split_L{L}", Hq, Hkv, D, [L], 256, 2048, 128, "keep_all", seed=L + 5)
    _parity(kvs, wl, wl.evict_at())
    t = inputs.make_tensors(wl)
    a = gpu_fwd_bwd(kvs, t["q"], t["k"], t["v"], t["do"], wl.evict_at(), wl.softmax_scale)
    b = gpu_fwd_bwd(kvs, t["q"], t["k"], t["v"], t["do"], wl.evict_at(), wl.softmax_scale)
    for key in ("dk", "dv"):
        assert torch.equal(a[key], b[key]), key


def test_long_key_spans_split_varlen(kvs):
    wl = inputs.custom_workload("split_varlen", 4, 2, 64, [700, 8500, 129], 300, 1500, 100, "last2", varlen=True,
                                seed=31)
    _parity(kvs, wl, wl.evict_at(), cu=wl.cu_seqlens())


# The re-prefill baseline (the fresh causal traces re-prefill compaction runs
# for the same rollout) goes through the same library as a varlen batch with
# nothing evicted.
@pytest.mark.parametrize("strategy", ["keep_all", "latest_only", "last2"])
def test_reprefill_batch(kvs, strategy):
    lengths = [len(t) for t in inputs.reprefill_traces(700, 33, 97, 13, strategy)]
    wl = inputs.custom_workload(f"reprefill_{strategy}", 6, 2, 128, lengths, 0, 1, 0, varlen=True, seed=41)
    e = np.concatenate([np.full(L, L, dtype=np.int32) for L in lengths])
    _parity(kvs, wl, e, cu=wl.cu_seqlens())


# Turn-level strategies of Section 3 (sliding window, Markovian Thinker,
# Markovian Pick), with and without 16-token turn padding: seeded random
# layouts (turn lengths, window, stride, picks, head grouping, D), each checked
# element by element.  Unaligned turn boundaries make most issued tiles PARTIAL.
def _turn_fuzz_case(seed):
    rng = np.random.default_rng(1000 + seed)
    strategy = inputs.TURN_STRATEGIES[seed % 3]
    window = int(rng.integers(3, 9))
    stride = int(rng.integers(1, window + 1))
    keep = int(rng.integers(0, window))
    lo = int(rng.integers(1, 40))
    hi = lo + int(rng.integers(0, 150))
    pad = 16 if seed % 2 else 1
    L = int(rng.integers(300, 1500))
    p = int(rng.integers(0, 100))
    Hq, Hkv = [(4, 4), (8, 2), (6, 3), (10, 2), (8, 1)][seed % 5]
    D = 128 if seed % 3 != 2 else 64
    return L, p, Hq, Hkv, D, (strategy, window, stride, keep, lo, hi, pad, 2000 + seed)


@pytest.mark.parametrize("seed", range(9))
def test_turn_strategy_fuzz(kvs, seed):
    L, p, Hq, Hkv, D, turns = _turn_fuzz_case(seed)
    wl = inputs.custom_workload(f"turns_{turns[0]}_{seed}", Hq, Hkv, D, [L], p, 0, 0, seed=3000 + seed, turns=turns)
    _parity(kvs, wl, wl.evict_at())


def test_turn_strategy_varlen(kvs):
    turns = ("markovian_pick", 5, 1, 2, 10, 90, 16, 77)
    wl = inputs.custom_workload("turns_varlen", 8, 2, 128, [513, 1, 700, 64], 20, 0, 0, varlen=True, seed=78,
                                turns=turns)
    _parity(kvs, wl, wl.evict_at(), cu=wl.cu_seqlens())


def test_self_only_closed_form(kvs):
    # every key lives for one query: O_i = v_i, dQ = dK = 0, dV_j = sum over the group of dO_j
    L, Hq, Hkv, D = 200, 4, 2, 128
    wl = inputs.custom_workload("self_only", Hq, Hkv, D, [L], 0, 1, 0, seed=77)
    t = inputs.make_tensors(wl)
    e = np.arange(1, L + 1, dtype=np.int32)
    announce("self_only closed form")
    res = gpu_fwd_bwd(kvs, t["q"], t["k"], t["v"], t["do"], e, 0.1)
    v = t["v"].double().numpy()
    G = Hq // Hkv
    for h in range(Hq):
        assert_flat("O", to_f64(res["O"][:, h]), v[:, h // G], max_abs=1e-6, rel_l2=1e-6)
    # dS = P (dP - Delta) vanishes up to the fp32 rounding of two sums of the same products
    assert float(res["dq"].abs().max()) < 1e-4 and float(res["dk"].abs().max()) < 1e-4
    ref_dv = t["do"].double().numpy().reshape(L, Hkv, G, D).sum(2)
    assert_close("dV", to_f64(res["dv"]), ref_dv, rel_l2=5e-3)


def test_forward_is_deterministic(kvs):
    wl = inputs.custom_workload("det", 8, 2, 128, [900], 64, 200, 50, "last2", seed=21)
    t = inputs.make_tensors(wl)
    announce("determinism")
    a = gpu_fwd_bwd(kvs, t["q"], t["k"], t["v"], t["do"], wl.evict_at(), wl.softmax_scale)
    b = gpu_fwd_bwd(kvs, t["q"], t["k"], t["v"], t["do"], wl.evict_at(), wl.softmax_scale)
    for key in ("O", "LSE", "dq", "dk", "dv"):
        assert torch.equal(a[key], b[key]), key


@pytest.mark.parametrize("BM,BN", [(32, 64), (64, 64), (128, 128), (96, 64), (32, 32), (16, 128), (128, 64)])
def test_tile_classes_exact(kvs, BM, BN):
    rng = np.random.default_rng(BM * 7 + BN)
    announce(f"classify BM={BM} BN={BN}")
    dev = torch.device("cuda:0")
    for L in (1, 31, 64, 65, 200, 777):
        for e in (inputs.evict_at_random(L, rng), inputs.evict_at_layout(L, 5, 40, 9, "last2"),
                  np.full(L, np.iinfo(np.int32).max, dtype=np.int32)):
            ev = torch.from_numpy(np.ascontiguousarray(e, dtype=np.int32)).to(dev)
            got = kvs.kvs_classify_tiles(ev.view(1, L), BM, BN).cpu().numpy()
            want = otiles.tile_classes(np.asarray(e), L, BM, BN).ravel()
            np.testing.assert_array_equal(got, want)
    # varlen packing, including an empty trace
    lens = [65, 0, 200, 1, 130]
    e = np.concatenate([inputs.evict_at_random(L, rng) for L in lens if L])
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device=dev)
    got = kvs.kvs_classify_tiles(torch.from_numpy(e).to(dev), BM, BN, cu_seqlens=cu).cpu().numpy()
    np.testing.assert_array_equal(got, otiles.tile_classes_packed(e, lens, BM, BN))


def test_tile_classes_of_workloads(kvs):
    dev = torch.device("cuda:0")
    for name in ("trace16k_gqa4", "trace64k_last2"):
        wl = inputs.WORKLOADS[name]
        e = wl.evict_at()
        L = wl.lengths[0]
        announce(f"classify {name}")
        got = kvs.kvs_classify_tiles(torch.from_numpy(e).to(dev).view(1, L), 128, 128).cpu().numpy()
        want = otiles.tile_classes(e, L, 128, 128).ravel()
        np.testing.assert_array_equal(got, want)


def test_check_evict_at(kvs):
    dev = torch.device("cuda:0")
    announce("check_evict_at")
    e = inputs.evict_at_layout(500, 10, 50, 5, "keep_all")
    ev = torch.from_numpy(e).to(dev)
    assert kvs.kvs_check_evict_at(ev.view(1, 500)) == -1
    bad = e.copy()
    bad[321] = 321
    bad[400] = 3
    assert kvs.kvs_check_evict_at(torch.from_numpy(bad).to(dev).view(1, 500)) == 321
    lens = [100, 400]
    cu = torch.tensor([0, 100, 500], dtype=torch.int32, device=dev)
    e2 = np.concatenate([inputs.evict_at_layout(100, 1, 9, 1), inputs.evict_at_layout(400, 3, 20, 2)])
    assert kvs.kvs_check_evict_at(torch.from_numpy(e2).to(dev), cu) == -1
    e2[150] = 50  # trace-local index 50 of trace 1: evict_at 50 <= 50
    assert kvs.kvs_check_evict_at(torch.from_numpy(e2).to(dev), cu) == 150
    badcu = torch.tensor([0, 300, 200], dtype=torch.int32, device=dev)
    with pytest.raises(kvs.KvsError):
        kvs.kvs_check_evict_at(torch.from_numpy(e2).to(dev), badcu)


def test_bench_mfma_rate_probe(kvs):
    announce("benchmark matrix-core probe")
    import bench

    rate = bench.measured_mfma_rate()
    # attainable dense bf16 rate on changing operands: positive and not above the published
    # 2516.6 TFLOP/s (2.4 GHz)
    assert 500.0 < rate <= 2516.6 * 1.02, rate
