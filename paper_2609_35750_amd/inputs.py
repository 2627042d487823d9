"""Seeded synthetic inputs for eviction-masked attention.

This module builds the two kinds of input that both the HIP path and the
CPU oracle consume, and nothing else: the per-key eviction index
``evict_at`` of a compacted agent trace, and seeded bf16 Q/K/V/dO tensors.
It holds none of the attention arithmetic.

Trace layout (Section 2, "KV-streams"; Section 3, "Summary"; Appendix B,
"Turn-Wise Compaction").  A trace of length ``L`` starts with a prompt
``[0, p)`` that is never evicted.  Segment ``k`` starts at ``a_k`` with
``a_0 = p`` and ``a_{k+1} = a_k + w + s``; it holds ``w`` turn tokens
``U_k = [a_k, a_k + w)`` followed by an ``s``-token summary
``S_k = [a_k + w, a_{k+1})`` (both clipped to ``[0, L)``).  Compaction ``k``
happens only once its summary is complete (``a_{k+1} <= L``): the summary is
generated while the turns are still visible, then the whole turns are
deleted, so ``evict_at[U_k] = a_{k+1}``.  Turns of a segment whose summary is
cut off by the end of the trace are never evicted.

Summary retention strategies:

* ``keep_all``     every summary stays for the rest of the trace;
* ``latest_only``  summary ``S_k`` is deleted when ``S_{k+1}`` completes,
                   i.e. ``evict_at[S_k] = a_{k+2}``;
* ``last2``        only the two newest summaries stay: ``S_k`` is deleted
                   when ``S_{k+2}`` completes, ``evict_at[S_k] = a_{k+3}``.

A key that is never evicted carries ``evict_at = L`` (any value ``>= L``
means the same).  Query ``i`` sees key ``j`` iff ``j <= i < evict_at[j]``.

Tensor recipe: fp32 standard normal draws from a seeded CPU
``torch.Generator`` (one seed per tensor), rounded to bf16 with
round-to-nearest-even.  Where a workload states that Q is pre-scaled by
``1/sqrt(D)``, Q is drawn as ``N(0,1)/sqrt(D)`` before rounding and the
softmax scale is 1.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np

STRATEGIES = ("keep_all", "latest_only", "last2")


def segment_starts(L: int, p: int, w: int, s: int) -> List[int]:
    """Start positions ``a_0, a_1, ...`` of every segment that begins before ``L``,
    plus one more start past the last one (so ``a_{k+1}`` always exists)."""
    if w + s <= 0:
        raise ValueError("segment length w + s must be positive")
    a = [p]
    while a[-1] < L:
        a.append(a[-1] + w + s)
    a.append(a[-1] + w + s)
    return a


def evict_at_layout(L: int, p: int, w: int, s: int, strategy: str = "keep_all") -> np.ndarray:
    """``evict_at`` (int32, length ``L``) of one trace built from the segment layout."""
    if strategy not in STRATEGIES:
        raise ValueError(f"unknown strategy {strategy!r}")
    if L < 0 or p < 0 or w < 0 or s < 0:
        raise ValueError("bad layout")
    if L == 0:  # an empty trace of a varlen batch
        return np.zeros(0, dtype=np.int32)
    e = np.full(L, L, dtype=np.int64)
    a = segment_starts(L, p, w, s)
    nseg = len(a) - 2

    def fired(k: int) -> bool:  # compaction k happens iff its summary completes inside the trace
        return 0 <= k < nseg and a[k + 1] <= L

    for k in range(nseg):
        if fired(k):
            e[a[k]:min(a[k] + w, L)] = a[k + 1]
        lo, hi = a[k] + w, min(a[k + 1], L)
        if lo >= hi:
            continue
        if strategy == "latest_only" and fired(k + 1):
            e[lo:hi] = a[k + 2]
        elif strategy == "last2" and fired(k + 2):
            e[lo:hi] = a[k + 3]
    return np.minimum(e, L).astype(np.int32)


# ---------------------------------------------------------------- turn-level strategies
# Section 3 ("Markovian Thinker", "Markovian Pick", "Sliding Window") and
# Appendix B ("Turn-Wise Compaction"): the context holds a prompt (never
# evicted) and whole turns; compaction removes whole turns and generates no
# summary.  Turn ``t`` occupies tokens ``[b_t, b_{t+1})`` with ``b_0 = p``.
# With a budget of ``window`` turns, a compaction fires right before a new
# turn would make the context exceed the budget:
#
# * ``sliding_window``     deletes the oldest ``stride`` turns (Section 3 uses
#                          stride 1 in the SFT masks, Section 4.3);
# * ``markovian_thinker``  deletes the oldest half (stride ``window // 2``);
# * ``markovian_pick``     keeps a chosen subset of ``keep`` turns and
#                          deletes the others (the choices are an input).
TURN_STRATEGIES = ("sliding_window", "markovian_thinker", "markovian_pick")


def turn_lengths(n: int, lo: int, hi: int, rng: np.random.Generator, pad: int = 1) -> List[int]:
    """``n`` turn lengths uniform on ``[lo, hi]``, each rounded up to a multiple of
    ``pad`` (16 mirrors the engine's 16-token KV blocks, Section 4)."""
    x = rng.integers(lo, hi, n, endpoint=True)
    return [int(-(-int(v) // pad) * pad) for v in x]


def pick_turns(n_turns: int, window: int, keep: int, rng: np.random.Generator) -> List[np.ndarray]:
    """Random Markovian Pick choices: for every compaction of a rollout of
    ``n_turns`` turns, the sorted positions (in the current context, oldest
    first) of the ``keep`` turns that stay."""
    if not 0 <= keep < window:
        raise ValueError("keep must be in [0, window)")
    picks, live = [], 0
    for _ in range(n_turns):
        if live == window:
            picks.append(np.sort(rng.choice(window, size=keep, replace=False)))
            live = keep
        live += 1
    return picks


def evict_at_turns(p: int, lengths: Sequence[int], strategy: str, window: int, stride: int = 1,
                   picks: Optional[Sequence[np.ndarray]] = None) -> np.ndarray:
    """``evict_at`` (int32, length ``p + sum(lengths)``) of a turn-level compaction."""
    if strategy not in TURN_STRATEGIES:
        raise ValueError(f"unknown turn strategy {strategy!r}")
    if window < 1 or any(x < 1 for x in lengths):
        raise ValueError("bad turn layout")
    n = len(lengths)
    b = np.concatenate([[p], p + np.cumsum(lengths)]).astype(np.int64)   # b[t] = first token of turn t
    L = int(b[-1])
    e = np.full(L, L, dtype=np.int64)
    if strategy in ("sliding_window", "markovian_thinker"):
        st = max(window // 2, 1) if strategy == "markovian_thinker" else stride
        if not 1 <= st <= window:
            raise ValueError("stride must be in [1, window]")
        # Turn t belongs to deletion group t // st; that group goes with the compaction before turn
        # (t // st) * st + window (the first turn that would overflow the budget with it still live).
        for t in range(n):
            gone = (t // st) * st + window
            if gone < n:
                e[b[t]:b[t + 1]] = b[gone]
    else:
        if picks is None:
            raise ValueError("markovian_pick needs the picks")
        live, c = [], 0
        for t in range(n):
            if len(live) == window:
                kept = [live[i] for i in picks[c]]
                for u in live:
                    if u not in kept:
                        e[b[u]:b[u + 1]] = b[t]
                live, c = kept, c + 1
            live.append(t)
    return np.minimum(e, L).astype(np.int32)


def turn_trace(L: int, p: int, strategy: str, window: int, stride: int, keep: int, lo: int, hi: int, pad: int,
               seed: int, trace: int = 0):
    """One trace of exactly ``L`` tokens under a turn-level strategy: turn lengths
    drawn from ``numpy.random.default_rng([seed, trace])`` (the last turn cut at
    ``L``), picks drawn from the same generator.  Returns ``(evict_at, lengths, picks)``."""
    rng = np.random.default_rng([seed, trace])
    lengths, tot = [], p
    while tot < L:
        x = turn_lengths(1, lo, hi, rng, pad=pad)[0]
        x = min(x, L - tot)
        lengths.append(x)
        tot += x
    if not lengths:
        return np.full(L, L, dtype=np.int32), [], None
    picks = pick_turns(len(lengths), window, keep, rng) if strategy == "markovian_pick" else None
    return evict_at_turns(min(p, L), lengths, strategy, window, stride=stride, picks=picks), lengths, picks


def reprefill_traces(L: int, p: int, w: int, s: int, strategy: str = "keep_all") -> List[np.ndarray]:
    """The fresh traces that re-prefill compaction runs for the same rollout
    (Section 2, "Prefill-compaction"; Appendix E).

    Without KV-streams every compaction continues in a new trace that first
    re-processes the entries the compaction keeps (the prompt and the retained
    summaries, with reset positions) and then holds the next segment.  Trace 0
    is the prompt plus segment 0; trace ``k >= 1`` is the prompt, the summaries
    retained by compaction ``k - 1`` under the strategy, then segment ``k``
    (clipped at ``L``).  Every trace is plain causal attention.  Returns, per
    trace, the original token index of each position.
    """
    if strategy not in STRATEGIES:
        raise ValueError(f"unknown strategy {strategy!r}")
    if L <= p or w + s <= 0:
        return [np.arange(L, dtype=np.int64)]
    a = segment_starts(L, p, w, s)
    prompt = np.arange(p, dtype=np.int64)
    traces = []
    k = 0
    while a[k] < L:
        new = np.arange(a[k], min(a[k + 1], L), dtype=np.int64)
        if k == 0:
            traces.append(np.concatenate([prompt, new]))
        else:
            if strategy == "keep_all":
                keep = range(0, k)
            elif strategy == "latest_only":
                keep = range(k - 1, k)
            else:
                keep = range(max(k - 2, 0), k)
            summ = [np.arange(a[c] + w, a[c + 1], dtype=np.int64) for c in keep]
            traces.append(np.concatenate([prompt] + summ + [new]))
        if a[k + 1] > L:   # the last segment's summary is cut off: no further compaction
            break
        k += 1
    return traces


def reprefill_traces_from_evict(e: np.ndarray) -> List[np.ndarray]:
    """Re-prefill traces of any single-trace eviction layout: every distinct
    eviction time ``t < L`` is a compaction; the fresh trace it opens first
    re-processes the entries generated before ``t`` that are still live after
    it (``e_j > t``) and then holds the tokens up to the next compaction."""
    e = np.asarray(e, dtype=np.int64)
    L = len(e)
    events = np.unique(e[e < L])
    events = events[events > 0]
    bounds = [0] + events.tolist() + [L]
    traces = [np.arange(0, bounds[1], dtype=np.int64)]
    for k in range(1, len(bounds) - 1):
        t = bounds[k]
        kept = np.nonzero(e[:t] > t)[0]
        traces.append(np.concatenate([kept, np.arange(t, bounds[k + 1], dtype=np.int64)]))
    return traces


def reprefill_extra_tokens(L: int, p: int, w: int, s: int, strategy: str = "keep_all") -> dict:
    """Extra prefilled entries of re-prefill compaction: the exact count for the
    layout (sum of the trace lengths minus ``L``) and the estimate
    ``N r / (B - r)`` of Section 2 (Appendix E), taking ``N = L - p`` generated
    entries, ``B - r = w + s`` new entries between compactions and ``r`` the
    mean number of kept entries over the traces that re-prefill them."""
    tr = reprefill_traces(L, p, w, s, strategy)
    exact = int(sum(len(t) for t in tr)) - L
    kept = []
    a = segment_starts(L, p, w, s) if L > p and w + s > 0 else [p]
    for k in range(1, len(tr)):
        kept.append(len(tr[k]) - (min(a[k + 1], L) - a[k]))
    r = float(np.mean(kept)) if kept else 0.0
    formula = (L - p) * r / (w + s) if kept else 0.0
    return {"traces": len(tr), "tokens": int(sum(len(t) for t in tr)), "extra_exact": exact,
            "kept_mean": r, "extra_formula": formula}


def evict_at_random(L: int, rng: np.random.Generator, p_never: float = 0.3) -> np.ndarray:
    """Unstructured valid eviction indices: ``e_j`` uniform on ``(j, L]`` (``L`` = never)."""
    e = np.empty(L, dtype=np.int64)
    for j in range(L):
        e[j] = L if rng.random() < p_never else rng.integers(j + 1, L + 1)
    return e.astype(np.int32)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload shaped like an agent trace batch."""

    name: str
    Hq: int
    Hkv: int
    D: int
    lengths: tuple
    p: int
    w: int
    s: int
    strategy: str
    q_prescaled: bool
    varlen: bool
    seed: int
    # Turn-level layout instead of (w, s) segments: (strategy, window, stride, keep, lo, hi, pad, seed).
    turns: Optional[tuple] = None

    @property
    def B(self) -> int:
        return len(self.lengths)

    @property
    def T(self) -> int:
        return max(self.lengths)

    @property
    def ntok(self) -> int:
        return int(sum(self.lengths))

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def softmax_scale(self) -> float:
        return 1.0 if self.q_prescaled else 1.0 / math.sqrt(self.D)

    def evict_at(self) -> np.ndarray:
        """Trace-local eviction indices, concatenated in trace order (int32, ``[ntok]``)."""
        if self.turns is not None:
            return np.concatenate([turn_trace(L, self.p, *self.turns, trace=b)[0] for b, L in enumerate(self.lengths)])
        return np.concatenate([evict_at_layout(L, self.p, self.w, self.s, self.strategy) for L in self.lengths])

    def cu_seqlens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.lengths)]).astype(np.int32)


def varlen_lengths(n: int, lo: int, hi: int, seed: int) -> tuple:
    """Trace lengths drawn i.i.d. uniform on ``[lo, hi]`` (inclusive) from a seeded numpy generator."""
    return tuple(int(x) for x in np.random.default_rng(seed).integers(lo, hi, n, endpoint=True))


def _workloads() -> Dict[str, Workload]:
    W = Workload
    return {
        w.name: w
        for w in [
            W("trace512_tiny", 4, 4, 64, (512,), 64, 128, 32, "keep_all", False, False, 1001),
            W("trace16k_gqa4", 32, 8, 128, (16384,), 1024, 4096, 512, "keep_all", True, False, 1002),
            W("trace32k_latest", 32, 8, 128, (32768,), 1024, 3072, 256, "latest_only", False, False, 1003),
            W("varlen8_gqa5", 40, 8, 128, varlen_lengths(8, 4096, 24576, 39), 512, 2048, 256, "keep_all", False, True, 1004),
            W("trace64k_last2", 64, 8, 128, (65536,), 2048, 2048, 256, "last2", False, False, 1005),
            # turn-level sliding window (TextWorld-like: 32k tokens, window of 10 turns, stride 1, turns of
            # 64..1024 tokens padded to 16)
            W("textworld32k_sliding", 32, 8, 128, (32768,), 1024, 0, 0, "sliding_window", False, False, 1006,
              ("sliding_window", 10, 1, 0, 64, 1024, 16, 1006)),
        ]
    }


WORKLOADS: Dict[str, Workload] = _workloads()
WORKLOAD_ORDER = ["trace512_tiny", "trace16k_gqa4", "trace32k_latest", "varlen8_gqa5", "trace64k_last2"]


def custom_workload(name: str, Hq: int, Hkv: int, D: int, lengths: Sequence[int], p: int, w: int, s: int,
                    strategy: str = "keep_all", q_prescaled: bool = False, varlen: Optional[bool] = None,
                    seed: int = 0, turns: Optional[tuple] = None) -> Workload:
    if varlen is None:
        varlen = len(lengths) > 1 and len(set(lengths)) > 1
    return Workload(name, Hq, Hkv, D, tuple(int(x) for x in lengths), p, w, s, strategy, q_prescaled, varlen, seed,
                    turns)


def randn_bf16(shape, seed: int, scale: float = 1.0):
    """bf16 tensor of ``N(0,1) * scale`` draws (fp32 draw, one rounding to bf16), on the CPU."""
    import torch

    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    x = torch.randn(*shape, generator=g, dtype=torch.float32)
    if scale != 1.0:
        x = x * scale
    return x.to(torch.bfloat16)


def make_tensors(wl: Workload, with_grad: bool = True):
    """Seeded bf16 CPU tensors ``q, k, v`` (and ``do``) for a workload.

    Packed layout ``[ntok, H, D]``; a fixed-length batch of ``B`` traces of
    length ``T`` is the same memory as ``[B, T, H, D]``.
    """
    n = wl.ntok
    qs = 1.0 / math.sqrt(wl.D) if wl.q_prescaled else 1.0
    out = {
        "q": randn_bf16((n, wl.Hq, wl.D), wl.seed * 16 + 1, qs),
        "k": randn_bf16((n, wl.Hkv, wl.D), wl.seed * 16 + 2),
        "v": randn_bf16((n, wl.Hkv, wl.D), wl.seed * 16 + 3),
    }
    if with_grad:
        out["do"] = randn_bf16((n, wl.Hq, wl.D), wl.seed * 16 + 4)
    return out

