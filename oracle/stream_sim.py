"""Brute-force replay of a streamed, compacted KV cache (test infrastructure).

This is the inference-side picture of Section 2: a rollout appends one
(k, v) entry per token to a live cache; when a compaction fires, the delete
operator removes whole turns (Appendix B, "Turn-Wise Compaction") and the
summary the model just generated stays (Section 3, "Summary"), keeping its
original cache entry instead of being prefilled again ("KV-streams"
paragraph).  Each query attends over exactly the entries that are live when
it is generated.

The replay works from the strategy's description only, not from any
``evict_at`` array: the trace is a prompt of ``p`` tokens, then segments of
``w`` turn tokens followed by an ``s``-token summary.  When the summary of
segment k is complete (i.e. just before the first token of segment k+1), the
cache drops every turn token of segment k, and, depending on the strategy,
old summaries:

* ``keep_all``     none;
* ``latest_only``  every summary except the one just completed;
* ``last2``        every summary except the two newest.

It is used to pin both the masked one-pass definition and the layout rules
that produce ``evict_at``.  torch fp64 (autograd gives the gradients).
"""
from __future__ import annotations

import numpy as np


def replay(q, k, v, p: int, w: int, s: int, strategy: str, scale: float, return_live: bool = False):
    """Attend each query over the live cache of a single trace.

    ``q`` [L,Hq,D], ``k``/``v`` [L,Hkv,D] torch fp64 tensors (may require grad).
    Returns ``O`` [L,Hq,D] and ``LSE`` [Hq,L] (torch), and optionally the list of
    live key index sets, one per query.
    """
    import torch

    L, Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    seg_len = w + s
    live = []          # (token index, role, segment) of every live cache entry
    outs, lses, lives = [], [], []
    for t in range(L):
        # A compaction completes right before the first token of the next segment.
        if t > p and seg_len > 0 and (t - p) % seg_len == 0:
            done = (t - p) // seg_len - 1          # segment whose summary just completed
            kept = []
            for (j, role, seg) in live:
                if role == "turn" and seg == done:
                    continue                        # delete: whole turns of that segment
                if role == "summary":
                    if strategy == "latest_only" and seg < done:
                        continue
                    if strategy == "last2" and seg < done - 1:
                        continue
                kept.append((j, role, seg))
            live = kept
        if t < p:
            role, seg = "prompt", -1
        else:
            seg = (t - p) // seg_len
            role = "turn" if (t - p) % seg_len < w else "summary"
        live.append((t, role, seg))
        idx = torch.tensor([j for (j, _, _) in live], dtype=torch.long)
        lives.append(idx.numpy().copy())
        heads_o, heads_l = [], []
        for h in range(Hq):
            g = h // G
            sc = scale * (k[idx, g, :] @ q[t, h, :])
            lse = torch.logsumexp(sc, dim=0)
            heads_o.append(torch.softmax(sc, dim=0) @ v[idx, g, :])
            heads_l.append(lse)
        outs.append(torch.stack(heads_o))
        lses.append(torch.stack(heads_l))
    O = torch.stack(outs)
    LSE = torch.stack(lses).T
    if return_live:
        return O, LSE, lives
    return O, LSE


def live_sets_to_evict_at(lives, L: int) -> np.ndarray:
    """The eviction index each key would need so that one masked pass sees
    exactly the replayed live sets: the first query after which the key is gone."""
    e = np.full(L, L, dtype=np.int64)
    present = np.zeros(L, dtype=bool)
    for t, idx in enumerate(lives):
        now = np.zeros(L, dtype=bool)
        now[idx] = True
        gone = present & ~now
        e[gone & (e == L)] = t
        if np.any(now & ~present & (np.arange(L) != t)):
            raise AssertionError("a deleted key came back")
        present = now
    return e


def live_sets_turns(p: int, lengths, strategy: str, window: int, stride: int = 1, picks=None):
    """Live cache of a turn-level compaction (Section 3; Appendix B), replayed
    token by token from the strategy's description: the cache holds the prompt
    and whole turns; right before the first token of a turn that would bring
    the context above ``window`` turns, a compaction deletes whole turns:

    * ``sliding_window``     the ``stride`` oldest turns;
    * ``markovian_thinker``  the oldest half (``window // 2`` turns);
    * ``markovian_pick``     every turn except the chosen ones (``picks[c]``:
                             positions, oldest first, of the turns kept at
                             compaction ``c``).

    Returns one sorted array of live token indices per query token."""
    turns = []     # live turns, oldest first: (turn id, [token indices])
    prompt = list(range(p))
    lives = [np.arange(t + 1) for t in range(p)]
    tok, comp = p, 0
    for t, n in enumerate(lengths):
        if len(turns) + 1 > window:
            if strategy == "sliding_window":
                turns = turns[stride:]
            elif strategy == "markovian_thinker":
                turns = turns[max(window // 2, 1):]
            elif strategy == "markovian_pick":
                turns = [turns[i] for i in picks[comp]]
            else:
                raise ValueError(strategy)
            comp += 1
        turns.append((t, []))
        for _ in range(n):
            turns[-1][1].append(tok)
            live = prompt + [j for (_, toks) in turns for j in toks]
            lives.append(np.array(sorted(live), dtype=np.int64))
            tok += 1
    return lives


def attend_live(q, k, v, lives, scale: float):
    """O [L,Hq,D] and LSE [Hq,L] (torch) of each query over its live key set."""
    import torch

    L, Hq, D = q.shape
    G = Hq // k.shape[1]
    outs, lses = [], []
    for t in range(L):
        idx = torch.as_tensor(lives[t], dtype=torch.long)
        ho, hl = [], []
        for h in range(Hq):
            sc = scale * (k[idx, h // G, :] @ q[t, h, :])
            hl.append(torch.logsumexp(sc, dim=0))
            ho.append(torch.softmax(sc, dim=0) @ v[idx, h // G, :])
        outs.append(torch.stack(ho))
        lses.append(torch.stack(hl))
    return torch.stack(outs), torch.stack(lses).T
