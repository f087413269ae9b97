"""Pins for the matched-compute arms of the oracle (Sec. 3.3: token- and channel-level
partial forwarding, whole-timestep recomputation), by the cases that reduce to FeatFix,
Verify or Vanilla."""
import numpy as np
import pytest

import oracle as O
import synth


def tiny():
    cfg = synth.get_config("tiny")
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    return cfg, W, synth.make_inputs(cfg)


@pytest.mark.parametrize("mode", [O.TOKENS_PARTIAL, O.CHANNELS_PARTIAL])
def test_stride_one_partial_arm_is_featfix(mode):
    cfg, W, inp = tiny()
    mask = synth.site_mask(cfg)
    ff = O.run(cfg, O.FEATFIX, inp, W, mask)
    arm = O.run(cfg, mode, inp, W, mask, stride=1)
    assert np.array_equal(arm["x"], ff["x"])
    assert arm["counts"] == ff["counts"]


@pytest.mark.parametrize("mode,stride", [(O.TOKENS_PARTIAL, 2), (O.CHANNELS_PARTIAL, 2), (O.TOKENS_PARTIAL, 3),
                                         (O.CHANNELS_PARTIAL, 5)])
def test_first_site_mixes_exact_and_draft(mode, stride):
    # up to the first paid site every mode computes the same states, so the stream after
    # it is FeatFix's exact output on the chosen tokens / channels and Verify's draft on
    # the others
    cfg, W, inp = tiny()
    mask = synth.site_mask(cfg)
    L = len(cfg["kinds"])
    plan = O.make_plan(cfg["T"], L, cfg["R"], cfg["K"], cfg["S"], mask, O.FEATFIX)
    first = min((i, l) for i in range(cfg["T"]) for l in range(L) if plan["action"][i, l] == O.SITE)
    k = first[0] * L + first[1]
    tr = {m: [] for m in (O.FEATFIX, O.VERIFY, mode)}
    for m in tr:
        O.run(cfg, m, inp, W, mask, trace=tr[m], stride=stride)
    hf, hd, got = tr[O.FEATFIX][k], tr[O.VERIFY][k], tr[mode][k]
    assert not np.array_equal(hf, hd)
    sel = np.zeros(got.shape, bool)
    if mode == O.TOKENS_PARTIAL:
        sel[:, ::stride, :] = True
    else:
        sel[:, :, ::stride] = True
    assert np.array_equal(got[sel], hf[sel]) and np.array_equal(got[~sel], hd[~sel])


def test_recompute_from_layer_zero_is_vanilla():
    # a site at layer 0 of every cached step: the whole cached step is exact
    cfg, W, inp = tiny()
    T, L = cfg["T"], len(cfg["kinds"])
    mask = np.zeros((T, L), np.uint8)
    mask[:, 0] = 1
    rc = O.run(cfg, O.RECOMPUTE, inp, W, mask)
    va = O.run(cfg, O.VANILLA, inp, W, mask)
    assert np.array_equal(rc["x"], va["x"])
    cached = sum(1 for i in range(T) if i % cfg["R"])
    assert rc["counts"]["n_paid_checks"] == cached and rc["counts"]["n_recomputed"] == cached * (L - 1)


def test_recompute_with_last_layer_sites_is_featfix():
    # nothing follows the last layer, so there is nothing to recompute
    cfg, W, inp = tiny()
    T, L = cfg["T"], len(cfg["kinds"])
    mask = np.zeros((T, L), np.uint8)
    mask[:, L - 1] = 1
    rc = O.run(cfg, O.RECOMPUTE, inp, W, mask)
    ff = O.run(cfg, O.FEATFIX, inp, W, mask)
    assert np.array_equal(rc["x"], ff["x"])
    assert rc["counts"] == ff["counts"]


def test_recompute_differs_from_featfix_with_a_middle_site():
    cfg, W, inp = tiny()
    mask = synth.site_mask(cfg)
    rc = O.run(cfg, O.RECOMPUTE, inp, W, mask)
    ff = O.run(cfg, O.FEATFIX, inp, W, mask)
    assert not np.array_equal(rc["x"], ff["x"])
    assert rc["counts"]["n_recomputed"] > 0
