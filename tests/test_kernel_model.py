"""The CPU model of the kernels' arithmetic (``tests/kernel_model.py``), and the
parity bound derived from it.

* The model is the oracle's computation up to the kernels' roundings: it
  meets the stated bar (max |x - x*| <= 2e-2 where bf16 spacing allows it,
  relative L2 <= 1e-2) against the fp64 oracle.
* Replaying the forward's tile walk and its wave-wide rescale decision on a
  layout without a permanent prompt (Section 2 segments with p = 0: the first
  keys are evicted) shows why the rescale factor needs its guard: without it
  the rows that have seen no visible key when another row of their wave moves
  its maximum get exp2(-inf - -inf) = NaN; with it every output is finite.
* The parity bound of the GPU tests is |x - x*| <= 2e-2 + C ulp_bf16(x*)
  (+ 2^-8 E for dQ, below).  C comes from the model: the largest excess over
  the rest of the bound, in units of the bf16 spacing at x*, over workloads
  shaped like the benchmark configurations (scaled down so that the oracle
  finishes in seconds) must be at most C, and C at most twice that excess.
  The excess is the final rounding: a bf16 output between 8 and 16 is up to
  1/32 from the exact value, more than 2e-2.
* dQ = scale sum_j dS_ij k_j is a sum of terms much larger than the result.
  A backward that takes O in bf16 (as the API does) forms Delta from the
  rounded O, and a bf16 matrix-core product rounds every dS to bf16; both
  errors reach dQ multiplied by the softmax scale.  With the query pre-scaled
  by 1/sqrt(D) and scale 1 (the 16k workload), the model's dQ is up to 0.09
  off at elements far smaller than 4, i.e. no bf16 spacing at x* explains it.
  The dQ bound therefore adds the first-order effect of those two roundings,
  2^-8 E with E = oracle.attention.dq_rounding_scale (2^-8: the relative
  rounding error bound of bf16).
* dK and dV sum over the G q-heads of their group as well as over rows.  With
  G = 16 or 64 the rounded P, dS and O (through Delta) leave the model's dK
  and dV up to 1.5 times the bound above; the errors of the many independent
  roundings add like a random walk, so the dK/dV bound adds
  lambda 2^-8 S with S = oracle.attention.dkdv_rounding_rss (the root sum of
  squares of the rounded terms) and lambda = 7 (Hoeffding: at most 5e-11 per
  element); the model needs under a tenth of that.
"""
import numpy as np
import pytest

from oracle import attention as orc
from paper_2609_35750_amd import inputs
from tests import kernel_model as km
from tests.gpu_helpers import DQ_GAMMA, MAX_ABS, REL_L2, RSS_LAMBDA, U_BF16, ULP_FACTOR

KEYS = (("O", "O"), ("dQ", "dq"), ("dK", "dk"), ("dV", "dv"))

# Shaped like the benchmark configurations (GQA group, D, pre-scaled Q, strategy, varlen tails), scaled down.
CASES = {
    "trace512_tiny": inputs.WORKLOADS["trace512_tiny"],
    "like_16k_gqa4_prescaled": inputs.custom_workload("c2", 8, 2, 128, [1536], 128, 512, 64, "keep_all",
                                                      q_prescaled=True, seed=21),
    "like_32k_latest": inputs.custom_workload("c3", 8, 2, 128, [1536], 128, 384, 32, "latest_only", seed=22),
    "like_varlen_gqa5": inputs.custom_workload("c4", 10, 2, 128, [613, 931], 64, 256, 32, "keep_all", seed=23),
    "like_64k_last2_gqa8": inputs.custom_workload("c5", 16, 2, 128, [1536], 512, 256, 32, "last2", seed=41),
}


def _run(wl, guard=True):
    t = inputs.make_tensors(wl)
    e = wl.evict_at()
    cu = wl.cu_seqlens() if wl.varlen else None
    arrs = [t[x].float().numpy() for x in ("q", "k", "v", "do")]
    model = km.run(arrs[0], arrs[1], arrs[2], e, wl.softmax_scale, arrs[3], cu_seqlens=cu, guard=guard)
    return model, t, e, cu


def test_rounding_helpers():
    km.math_check()


@pytest.fixture(scope="module")
def emulated():
    out = {}
    for name, wl in CASES.items():
        model, t, e, cu = _run(wl)
        ref = orc.backward(t["q"], t["k"], t["v"], e, wl.softmax_scale, t["do"], cu_seqlens=cu)
        E = orc.dq_rounding_scale(t["q"], t["k"], t["v"], e, wl.softmax_scale, t["do"], np.arange(wl.ntok),
                                  cu_seqlens=cu)
        out[name] = (model, ref, E, wl)
    return out


def _flat(key, E):
    """The part of the bound that is not in units of the bf16 spacing at x*."""
    return MAX_ABS + (DQ_GAMMA * E if key == "dq" else 0.0)


def test_model_meets_the_stated_bar(emulated):
    for name, (model, ref, E, wl) in emulated.items():
        assert np.abs(model["LSE"] - ref["LSE"]).max() < 1e-5, name
        for label, key in KEYS:
            x, y = model[key], ref[key]
            rel = np.linalg.norm(x - y) / np.linalg.norm(y)
            assert rel <= REL_L2 / 2, (name, label, rel)
            # where the bf16 spacing is at most 2e-2, the flat bound holds for every output whose
            # softmax scale sits in the kernel (1/sqrt(D)); the pre-scaled query's dQ needs E
            small = km.ulp_bf16(y) <= MAX_ABS
            if key != "dq" or not wl.q_prescaled:
                assert np.abs(x - y)[small].max() <= MAX_ABS, (name, label)


def test_dq_needs_the_rounding_term_only_with_the_prescaled_query(emulated):
    for name, (model, ref, E, wl) in emulated.items():
        plain = km.excess_ulps(model["dq"], ref["dq"], MAX_ABS)
        if wl.q_prescaled:
            assert plain > 20.0, (name, plain)   # not explained by the spacing at x*
        else:
            assert plain <= ULP_FACTOR, (name, plain)
        # the first-order term is not vacuous: somewhere the model needs at least a quarter of it
        need = float(((np.abs(model["dq"] - ref["dq"]) - MAX_ABS) / (DQ_GAMMA * E)).max())
        if wl.q_prescaled:
            assert 0.25 < need <= 1.0, (name, need)


def test_parity_bound_constant_from_the_model(emulated):
    worst = 0.0
    table = []
    for name, (model, ref, E, wl) in emulated.items():
        for label, key in KEYS:
            x, y = model[key], ref[key]
            c = float((np.maximum(np.abs(x - y) - _flat(key, E), 0.0) / km.ulp_bf16(y)).max())
            worst = max(worst, c)
            table.append(f"{name}:{label} maxabs {np.abs(x - y).max():.4f} "
                         f"max|x*| {np.abs(y).max():.2f} excess {c:.3f} ulp")
    print("\n".join(table))
    print(f"largest excess: {worst:.3f} bf16 ulp; bound uses C = {ULP_FACTOR}")
    assert worst > 0.0, "some output must exceed the flat bound, else C is not needed"
    assert worst <= ULP_FACTOR <= 2.0 * worst


def test_unguarded_rescale_gives_nan_rows_and_guard_fixes_them():
    # No permanent prompt: the first segment's turns [0, 100) are evicted at 120, so rows 120..127
    # see nothing in the first key tile while rows 96..119 of the same wave do.
    for D in (64, 128):
        wl = inputs.custom_workload(f"p0_{D}", 4, 2, D, [1000], 0, 100, 20, "keep_all", seed=31)
        bad, _, _, _ = _run(wl, guard=False)
        rows = np.nonzero(~np.isfinite(bad["O"]).all(axis=(1, 2)))[0]
        assert rows.tolist() == list(range(120, 128)), (D, rows[:20])
        good, t, e, _ = _run(wl, guard=True)
        for key in ("O", "LSE", "dq", "dk", "dv"):
            assert np.isfinite(good[key]).all(), (D, key)
        ref = orc.forward(t["q"], t["k"], t["v"], e, wl.softmax_scale)
        assert np.abs(good["O"] - ref[0]).max() < MAX_ABS


# Large GQA groups (dK/dV sum 16 and 64 q-heads), scaled down.
GROUP_CASES = {
    "group16": inputs.custom_workload("g16", 32, 2, 128, [300], 9, 41, 7, "last2", seed=332),
    "group64": inputs.custom_workload("g64", 64, 1, 64, [200], 9, 41, 7, "last2", seed=264),
}


def test_dkdv_rounding_term_needed_for_large_groups_and_sufficient():
    for name, wl in GROUP_CASES.items():
        model, t, e, cu = _run(wl)
        ref = orc.backward(t["q"], t["k"], t["v"], e, wl.softmax_scale, t["do"], cu_seqlens=cu)
        SK, SV = orc.dkdv_rounding_rss(t["q"], t["k"], t["v"], e, wl.softmax_scale, t["do"], cu_seqlens=cu)
        worst_plain, worst_lam = 0.0, 0.0
        for key, S in (("dk", SK), ("dv", SV)):
            d = np.abs(model[key] - ref[key])
            plain = MAX_ABS + ULP_FACTOR * km.ulp_bf16(ref[key])
            worst_plain = max(worst_plain, float((d / plain).max()))
            lam = float((np.maximum(d - plain, 0.0) / (U_BF16 * S)).max())
            worst_lam = max(worst_lam, lam)
            print(f"{name}:{key} worst / plain bound {float((d / plain).max()):.3f}, lambda needed {lam:.3f}")
        assert worst_plain > 1.0, (name, worst_plain)          # the plain bound does not hold
        assert 0.0 < worst_lam <= RSS_LAMBDA / 10, (name, worst_lam)
