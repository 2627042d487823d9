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
