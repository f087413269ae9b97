"""Pins for classifier-free guidance by batch doubling in the oracle, and the ABI's checks
of the guidance fields.  Reading: the B model rows are B/2 conditional samples (rows b)
and their unconditional twins (rows B/2 + b); both rows of a pair read latent b and the
Euler step moves it by v_u + s (v_c - v_u)."""
import ctypes as C

import numpy as np
import pytest

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline


def guided(base="tiny", B=4, s=3.5, T=6, **kw):
    cfg = dict(synth.get_config(base, **kw))
    cfg.update(B=B, T=T, cfg_pairs=1, cfg_scale=s)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    return cfg, W, synth.make_inputs(cfg)


def rows(inp, sl, x=None):
    """The same inputs restricted to conditioning rows sl (x given or kept)."""
    return {"x": inp["x"] if x is None else x, "c": inp["c"][sl], "txt": inp["txt"][sl]}


def plain(cfg, B):
    c = dict(cfg)
    c.update(B=B, cfg_pairs=0)
    return c


MMDIT = dict(kinds=[synth.MMDIT_DOUBLE, synth.MMDIT_SINGLE], n_txt=8, sites=[1])


def test_inputs_hold_half_the_latents():
    cfg, _, inp = guided()
    assert inp["x"].shape[0] == 2 and inp["c"].shape[0] == 4


@pytest.mark.parametrize("kw", [{}, MMDIT], ids=["dit", "mmdit"])
def test_one_step_is_the_combination_of_two_plain_steps(kw):
    # one Euler step is linear in v: the guided latent equals x1_u + s (x1_c - x1_u) of an
    # unguided run over the same B rows whose latent batch is [x; x]
    cfg, W, inp = guided(T=1, **kw)
    half = cfg["B"] // 2
    mask = synth.site_mask(cfg)
    g = O.run(cfg, O.VANILLA, inp, W, mask)["x"]
    both = O.run(plain(cfg, cfg["B"]), O.VANILLA, rows(inp, slice(None), np.concatenate([inp["x"]] * 2)), W,
                 mask)["x"]
    xc, xu = both[:half], both[half:]
    np.testing.assert_allclose(g, xu + cfg["cfg_scale"] * (xc - xu), rtol=0, atol=1e-12 * np.abs(g).max())
    assert np.abs(xc - xu).max() > 1e-3        # the two conditionings do differ


@pytest.mark.parametrize("mode", [O.VANILLA, O.FEATFIX, O.VERIFY])
@pytest.mark.parametrize("kw", [{}, MMDIT], ids=["dit", "mmdit"])
def test_unit_and_zero_scale_are_the_single_branches(mode, kw):
    # s = 1 follows the conditional rows alone and s = 0 the unconditional rows alone,
    # over a whole cached loop (the fixed schedule keeps rows independent)
    for s, sl in ((1.0, slice(0, 2)), (0.0, slice(2, 4))):
        cfg, W, inp = guided(s=s, **kw)
        mask = synth.site_mask(cfg)
        g = O.run(cfg, mode, inp, W, mask)
        one = O.run(plain(cfg, 2), mode, rows(inp, sl), W, mask)
        np.testing.assert_allclose(g["x"], one["x"], rtol=0, atol=1e-10 * np.abs(one["x"]).max())
        # the audit covers all B rows; the branch's rows match the single run's
        for key, d in one["audit"].items():
            np.testing.assert_allclose(g["audit"][key][sl], d, rtol=1e-9, atol=1e-14)


def test_guidance_extrapolates_linearly_in_the_scale():
    # with one step the latent is affine in s: x(s) = x(0) + s (x(1) - x(0))
    out = {}
    for s in (0.0, 1.0, 4.0):
        cfg, W, inp = guided(T=1, s=s)
        out[s] = O.run(cfg, O.FEATFIX, inp, W, synth.site_mask(cfg))["x"]
    np.testing.assert_allclose(out[4.0], out[0.0] + 4.0 * (out[1.0] - out[0.0]), rtol=0,
                               atol=1e-11 * np.abs(out[4.0]).max())


@pytest.mark.parametrize("B,pairs,scale,code", [
    (3, 1, 2.0, abi.FF_E_SHAPE), (4, 2, 2.0, abi.FF_E_RANGE), (4, -1, 2.0, abi.FF_E_RANGE),
    (4, 1, float("nan"), abi.FF_E_RANGE), (4, 1, float("inf"), abi.FF_E_RANGE),
    (4, 1, 2.0, abi.FF_E_NULL), (3, 0, float("nan"), abi.FF_E_NULL)])
def test_guidance_descriptor_checks(B, pairs, scale, code):
    # the descriptor is checked before anything else of a call (NULL weights come after);
    # the scale is not read without pairs
    cfg = synth.get_config("tiny", B=B, cfg_pairs=pairs, cfg_scale=scale)
    m = pipeline.model_desc(cfg)
    got = abi.lib().ff_block_exact(C.byref(m), 0, None, None, None, None, None, 0, None)
    assert got == code, (B, pairs, scale, got)
