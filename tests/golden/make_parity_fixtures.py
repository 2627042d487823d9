"""Write the sampled expected outputs of the full-size workloads (CPU checker only).

    python tests/golden/make_parity_fixtures.py [workload ...]

For each workload the fp64 checker runs forward + backward for the q-heads of
KV head 0 over the whole workload (every trace, every row), and the script
stores, as float32:

* O, LSE, dQ of those q-heads at a set of sampled query rows that covers the
  prompt, every kind of segment boundary, summaries and the trace ends;
* dK, dV of KV head 0 at a set of sampled keys chosen the same way.

Inputs are the seeded synthetic tensors of ``paper_2609_35750_amd.inputs``;
the GPU test regenerates them and compares the library's outputs at the same
positions.  Nothing here reads anything the HIP library produced.
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import attention as orc  # noqa: E402
from paper_2609_35750_amd import inputs  # noqa: E402

N_SAMPLES = 96


def sample_positions(wl, rng):
    """Packed token indices: boundaries of the layout in every trace plus random fill."""
    picks = set()
    off = 0
    for b, L in enumerate(wl.lengths):
        marks = [0, 1, wl.p - 1, wl.p, L - 2, L - 1]
        if wl.turns is not None:   # turn boundaries
            _, lengths, _ = inputs.turn_trace(L, wl.p, *wl.turns, trace=b)
            for a in np.cumsum([wl.p] + list(lengths))[:-1]:
                marks += [a - 1, a, a + 1]
        else:
            starts = inputs.segment_starts(L, wl.p, wl.w, wl.s)
            for a in starts[:-1]:
                marks += [a - 1, a, a + 1, a + wl.w - 1, a + wl.w, a + wl.w + 1]
        for m in marks:
            if 0 <= m < L:
                picks.add(off + m)
        off += L
    picks = sorted(picks)
    if len(picks) > N_SAMPLES * 2 // 3:
        picks = sorted(rng.choice(picks, N_SAMPLES * 2 // 3, replace=False).tolist())
    rest = N_SAMPLES - len(picks)
    pool = np.setdiff1d(np.arange(wl.ntok), picks)
    picks += rng.choice(pool, rest, replace=False).tolist()
    return np.array(sorted(picks), dtype=np.int64)


def make(name):
    wl = inputs.WORKLOADS[name]
    t0 = time.time()
    t = inputs.make_tensors(wl)
    e = wl.evict_at()
    G = wl.G
    cu = wl.cu_seqlens() if wl.varlen else None
    res = orc.backward(t["q"][:, :G], t["k"][:, :1], t["v"][:, :1], e, wl.softmax_scale, t["do"][:, :G],
                       cu_seqlens=cu)
    rng = np.random.default_rng(7)
    rows = sample_positions(wl, rng)
    keys = sample_positions(wl, np.random.default_rng(8))
    out = {
        "rows": rows,
        "keys": keys,
        "heads": np.arange(G),
        "O": res["O"][rows].astype(np.float32),
        "LSE": res["LSE"][:, rows].astype(np.float32),
        "dQ": res["dq"][rows].astype(np.float32),
        "dK": res["dk"][keys, 0].astype(np.float32),
        "dV": res["dv"][keys, 0].astype(np.float32),
        # whole-tensor magnitudes of the group's outputs, for relative checks
        "norm_O": np.float64(np.linalg.norm(res["O"])),
        "norm_dQ": np.float64(np.linalg.norm(res["dq"])),
        "norm_dK": np.float64(np.linalg.norm(res["dk"])),
        "norm_dV": np.float64(np.linalg.norm(res["dv"])),
    }
    path = os.path.join(HERE, f"parity_{name}.npz")
    np.savez_compressed(path, **out)
    print(f"{name}: wrote {path} in {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    names = sys.argv[1:] or ["trace16k_gqa4", "trace32k_latest", "varlen8_gqa5", "trace64k_last2"]
    for n in names:
        make(n)
