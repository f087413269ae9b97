"""Pins for the adaptive (discrepancy-triggered) refresh policy of the oracle and the
ABI's checks of its threshold.  The policy reading: step 0 refreshes; step i refreshes
when R steps have passed since the last refresh, or when step i-1 was a cached step whose
largest paid-site discrepancy (Eq. 4) is not <= tau; finite differences use the actual
refresh steps (Eq. 2)."""
import math

import numpy as np
import pytest

import oracle as O
import synth
from paper_2607_27842_amd import abi


def tiny(T=9, R=3):
    cfg = dict(synth.get_config("tiny"))
    cfg["T"], cfg["R"] = T, R
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    return cfg, W, inp


@pytest.mark.parametrize("mode", [O.VERIFY, O.FEATFIX])
def test_huge_threshold_is_the_fixed_schedule(mode):
    # no discrepancy reaches 1e30: only the interval R refreshes, exactly as i % R == 0
    cfg, W, inp = tiny()
    mask = synth.site_mask(cfg)
    fixed = O.run(cfg, mode, inp, W, mask)
    adapt = O.run(cfg, mode, inp, W, mask, tau=1e30)
    assert adapt["step_kind"] == [O.REFRESH_STEP if i % cfg["R"] == 0 else O.CACHED_STEP for i in range(cfg["T"])]
    assert np.array_equal(adapt["x"], fixed["x"])
    assert adapt["counts"] == fixed["counts"] == fixed["plan"]["counts"]


@pytest.mark.parametrize("mode", [O.VERIFY, O.FEATFIX])
def test_tiny_threshold_refreshes_after_every_check(mode):
    # every cached step carries sites and any positive discrepancy exceeds 1e-30: the
    # steps alternate refresh / cached (the interval cap R = 3 never binds), which is the
    # fixed schedule with R = 2 -- the same refresh steps, hence the same arithmetic
    cfg, W, inp = tiny(T=9, R=3)
    mask = synth.site_mask(cfg)
    assert all(mask[i].any() for i in range(cfg["T"]))
    adapt = O.run(cfg, mode, inp, W, mask, tau=1e-30)
    assert adapt["step_kind"] == [O.REFRESH_STEP if i % 2 == 0 else O.CACHED_STEP for i in range(9)]
    assert all(float(np.min(d)) > 1e-30 for d in adapt["audit"].values())
    cfg2 = dict(cfg)
    cfg2["R"] = 2
    fixed2 = O.run(cfg2, mode, inp, W, mask)
    assert np.array_equal(adapt["x"], fixed2["x"])
    assert adapt["counts"] == fixed2["counts"]


def test_interval_cap_without_sites():
    # a mask with no sites gives no discrepancy: refreshes only every R steps
    cfg, W, inp = tiny(T=8, R=3)
    mask = np.zeros((cfg["T"], len(cfg["kinds"])), np.uint8)
    adapt = O.run(cfg, O.FEATFIX, inp, W, mask, tau=1e-30)
    assert adapt["step_kind"] == [O.REFRESH_STEP if i % 3 == 0 else O.CACHED_STEP for i in range(8)]
    assert adapt["counts"]["n_paid_checks"] == 0


def test_threshold_needs_a_discrepancy_mode():
    cfg, W, inp = tiny(T=4)
    mask = synth.site_mask(cfg)
    for mode in (O.VANILLA, O.DRAFT, O.EXACT_ONLY):
        with pytest.raises(ValueError):
            O.run(cfg, mode, inp, W, mask, tau=0.5)


@pytest.mark.parametrize("K", [1, 2, 3])
def test_forecast_exact_on_linear_trajectories_with_uneven_gaps(K):
    # refreshes at steps 0, 2, 5, 6 (gaps 2, 3, 1): the divided differences of a linear
    # trajectory are its slope and zeros, so every forecast is exact
    a, b = np.array([0.5, -2.0]), np.array([1.25, 0.75])
    tc = O.TaylorCache(K)
    for tau in (0, 2, 5, 6):
        tc.refresh(a + b * tau, tau)
    for i in (7, 8, 11):
        np.testing.assert_allclose(tc.forecast(i), a + b * i, rtol=0, atol=1e-12)


def test_forecast_with_uneven_gaps_hand_computed():
    # K = 2, refreshes of f at 0, 1, 3 with f = t^2: D^0 = 9, D^1 = (9 - 1) / 2 = 4,
    # D^2 = (4 - 1) / 2 = 1.5 (the recursion divides by the latest gap only), so the
    # forecast at 4 is 9 + 4 + 1.5 / 2 = 13.75 against f(4) = 16
    tc = O.TaylorCache(2)
    for tau in (0, 1, 3):
        tc.refresh(np.array([float(tau * tau)]), tau)
    assert tc.forecast(4)[0] == 13.75


def sched(mode, tau, T=10, R=3, K=1, S=2):
    return abi.ff_sched_desc(T, R, K, S, 1e-8, mode, abi.FF_RESIDUAL, tau)


def test_abi_threshold_checks():
    L = 4
    mask = np.ones(10 * L, np.uint8)
    p = abi.ff_plan_build(sched(abi.FF_FEATFIX, 0.25), L, mask)
    abi.ff_plan_destroy(p)
    p = abi.ff_plan_build(sched(abi.FF_VERIFY, 0.25), L, mask)
    abi.ff_plan_destroy(p)
    for mode in (abi.FF_VANILLA, abi.FF_DRAFT, abi.FF_EXACT_ONLY):
        with pytest.raises(abi.FFError) as e:
            abi.ff_plan_build(sched(mode, 0.25), L, mask)
        assert e.value.status == abi.FF_E_RANGE
    for bad in (-1.0, math.inf, math.nan):
        with pytest.raises(abi.FFError) as e:
            abi.ff_plan_build(sched(abi.FF_FEATFIX, bad), L, mask)
        assert e.value.status == abi.FF_E_RANGE


def test_abi_threshold_plan_is_the_fixed_schedule():
    # the exported plan of an adaptive schedule is the one no discrepancy would change
    L, T, R = 4, 10, 3
    mask = np.ones(T * L, np.uint8)
    pa = abi.ff_plan_build(sched(abi.FF_FEATFIX, 0.25, T=T, R=R), L, mask)
    pf = abi.ff_plan_build(sched(abi.FF_FEATFIX, 0.0, T=T, R=R), L, mask)
    ea, ef = abi.ff_plan_export(pa, T, L, 1), abi.ff_plan_export(pf, T, L, 1)
    for k in ef:
        if k != "counts":
            np.testing.assert_array_equal(ea[k], ef[k])
    abi.ff_plan_destroy(pa)
    abi.ff_plan_destroy(pf)


def test_decision_takes_the_largest_discrepancy_over_samples():
    """B = 2 with a threshold that only sample 1's discrepancy exceeds at the first checked
    step: the step after it must refresh (the rule's maximum runs over sites and samples).
    tau sits above the mean of the two samples' maxima, so a reading that used sample 0
    only, or any mean over samples, would keep the step cached; run alone, sample 0 keeps
    it cached and sample 1 refreshes."""
    cfg, W, _ = tiny(T=9, R=4)
    cfg["B"] = 2
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    fixed = O.run(cfg, O.FEATFIX, inp, W, mask)
    first = min(i for (i, _l) in fixed["audit"])
    per_sample = np.max(np.stack([d for (i, _l), d in fixed["audit"].items() if i == first]), axis=0)
    if per_sample[0] > per_sample[1]:   # put the larger discrepancy on sample 1
        inp = {k: v[::-1].copy() for k, v in inp.items()}
        per_sample = per_sample[::-1]
    lo, hi = float(per_sample[0]), float(per_sample[1])
    assert hi > lo * 1.01, (lo, hi)
    tau = 0.5 * (0.5 * (lo + hi)) + 0.5 * hi      # in ((lo + hi) / 2, hi)
    both = O.run(cfg, O.FEATFIX, inp, W, mask, tau=tau)
    assert both["step_kind"][first + 1] == O.REFRESH_STEP
    alone = []
    for b in (0, 1):
        one = {k: v[b:b + 1] for k, v in inp.items()}
        r = O.run(dict(cfg, B=1), O.FEATFIX, one, W, mask, tau=tau)
        # the pair's audit of the first checked step is each sample's own (samples never mix)
        for (i, l), d in r["audit"].items():
            if i == first:
                np.testing.assert_allclose(d[0], both["audit"][(i, l)][b], rtol=1e-12)
        alone.append(r["step_kind"][first + 1])
    assert alone == [O.CACHED_STEP, O.REFRESH_STEP]
