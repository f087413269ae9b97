"""Loops whose conditioning is formed for the whole schedule at step 0 (ff_ctx_cond_cache):
c_t and every adaLN modulation vector depend on the class / text vector and the step only
(Eq. 1), so they are computed once per loop.  Checked against the oracle, for the bitwise
invariants of the mode definitions (Sec. 3.3), and for the host-side refusals."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import TOL, check_audit, host, need_gpu, say
from test_gpu_adaptive import pick_tau

pytestmark = pytest.mark.gpu

MODES = {"vanilla": abi.FF_VANILLA, "draft": abi.FF_DRAFT, "verify": abi.FF_VERIFY, "featfix": abi.FF_FEATFIX,
         "exact_only": abi.FF_EXACT_ONLY}
PLAN_KEYS = ("step_kind", "refresh_ord", "k_eff", "read_slots", "write_slot", "action")


def gpu_run(dm, cfg, inp, mode, mask, cond_cache=True, hist_sums=False, tau=0.0, R=None):
    r = pipeline.Runner(dm, mode, mask, cond_cache=cond_cache, hist_sums=hist_sums, tau=tau, R=R)
    assert (r.ccache is not None) == cond_cache
    x, c, txt = pipeline.host_inputs_to_device(cfg, inp)
    xt, audit, counts = r.run(x, c, txt)
    torch.cuda.synchronize()
    plan, kinds = r.export_plan(), list(r.step_kinds())
    r.close()
    return xt, audit, counts, plan, kinds


def against_oracle(cfg, W, inp, mode, mask, dm=None, hist_sums=False, label=""):
    dm = dm or pipeline.DeviceModel.from_host(cfg, *W)
    xt, audit, counts, plan, _ = gpu_run(dm, cfg, inp, mode, mask, hist_sums=hist_sums)
    ref = O.run(cfg, mode, inp, W, mask)
    err = O.max_rel_err(host(xt), ref["x"])
    say(f"{label}{cfg['name']} mode={mode} with the conditioning cache: max rel err {err:.3e}")
    assert err <= TOL[cfg["dtype"]], err
    assert counts == ref["counts"]
    for key in PLAN_KEYS:
        np.testing.assert_array_equal(plan[key], ref["plan"][key])
    check_audit(audit.cpu().numpy(), ref["audit"], cfg["dtype"], label=label)
    return xt


@pytest.mark.parametrize("mode", list(MODES))
def test_tiny_fp32_loop_with_cond_cache_matches_oracle(mode):
    """fp32: the modulation GEMMs over fp32 SiLU(c_t) rows."""
    need_gpu()
    cfg = synth.get_config("tiny")
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    against_oracle(cfg, W, inp, MODES[mode], synth.site_mask(cfg))


@pytest.mark.parametrize("B", [2, 11])
def test_tiny_bf16_loop_with_cond_cache_matches_oracle(B):
    """bf16: hi / lo rows of SiLU(c_t) through the GEMM, for one and for two groups of 8
    model rows (the second ragged)."""
    need_gpu()
    cfg = synth.get_config("tiny", dtype=synth.BF16, B=B, K=2, S=3, T=9)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    against_oracle(cfg, W, inp, abi.FF_FEATFIX, synth.site_mask(cfg))


def test_cond_cache_agrees_with_per_step_conditioning_fp32():
    """fp32: the cached and the per-step modulation differ only in fp32 summation order."""
    need_gpu()
    cfg = synth.get_config("tiny")
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    mask = synth.site_mask(cfg)
    a = gpu_run(dm, cfg, inp, abi.FF_FEATFIX, mask, cond_cache=True)
    b = gpu_run(dm, cfg, inp, abi.FF_FEATFIX, mask, cond_cache=False)
    err = O.max_rel_err(host(a[0]), host(b[0]))
    say(f"tiny fp32 cached vs per-step conditioning: max rel diff {err:.3e}")
    assert err <= 1e-6, err


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_cond_cache_keeps_the_bitwise_invariants(dtype):
    """FeatFix == Exact-only, Verify == Draft, all sites == Vanilla == R=1, repeat runs
    identical, with the conditioning cache (the per-layer step sets follow the mask, so
    these modes read identical modulation vectors)."""
    need_gpu()
    cfg = synth.get_config("tiny", dtype=dtype)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    mask = synth.site_mask(cfg)
    say(f"conditioning cache invariants dtype={dtype}")
    run = lambda mode, msk=mask, **kw: gpu_run(dm, cfg, inp, mode, msk, **kw)[0]
    ff, ff2 = run(abi.FF_FEATFIX), run(abi.FF_FEATFIX)
    assert torch.equal(ff, ff2)
    assert torch.equal(ff, run(abi.FF_EXACT_ONLY)), "FeatFix and Exact-only differ"
    assert torch.equal(run(abi.FF_VERIFY), run(abi.FF_DRAFT)), "Verify and Draft differ"
    va = run(abi.FF_VANILLA)
    assert torch.equal(run(abi.FF_FEATFIX, np.ones_like(mask)), va), "all-sites FeatFix differs from Vanilla"
    assert torch.equal(run(abi.FF_FEATFIX, R=1), va), "R=1 differs from Vanilla"


def test_dit_xl2_width_with_cond_cache_and_history_sums():
    """The bench's path at DiT-XL/2 width (C = 1152, 16 x 72 heads, 256 tokens, batch 8,
    bf16, K = 2), 4 blocks, T = 12 (k_eff = 2 at steps 10-11), sites {1, 3}: the non-site
    layers' modulation from the refresh steps' rows, the sites' from every step."""
    need_gpu()
    cfg = synth.get_config("dit_xl2", kinds=[synth.DIT] * 4, sites=[1, 3], T=12)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    against_oracle(cfg, W, inp, abi.FF_FEATFIX, synth.site_mask(cfg), hist_sums=True, label="DiT width: ")


def test_mmdit_with_cond_cache_matches_oracle():
    """MMDiT double (two weight sets per layer, 12C vectors) and single (3C) blocks with
    text rows: 2 double + 3 single, sites on the last double and the middle single."""
    need_gpu()
    C, H = 256, 2
    cfg = synth.get_config("flux", kinds=[synth.MMDIT_DOUBLE] * 2 + [synth.MMDIT_SINGLE] * 3, C=C, H=H, d=C // H,
                           mlp=4 * C, n_txt=24, lat=(16, 1, 20, 18), n_img=90, T=8, R=3, sites=[1, 3])
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    for mode in (abi.FF_FEATFIX, abi.FF_VERIFY):
        against_oracle(cfg, W, inp, mode, synth.site_mask(cfg), dm=dm, label="MMDiT: ")


def test_adaptive_with_cond_cache_takes_the_oracles_decisions():
    """tau > 0: every layer's modulation for every step; the realised schedule and latent
    equal the oracle's at a threshold that gives a mixed schedule with a clear margin."""
    need_gpu()
    cfg = synth.get_config("tiny", T=10, R=4)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    tau, ref = pick_tau(cfg, W, inp, O.FEATFIX, mask)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    xt, audit, counts, _plan, kinds = gpu_run(dm, cfg, inp, abi.FF_FEATFIX, mask, tau=tau)
    say(f"adaptive with the conditioning cache: tau {tau:.4e}, oracle kinds {ref['step_kind']}, GPU {kinds}")
    assert kinds == ref["step_kind"]
    assert counts == ref["counts"]
    err = O.max_rel_err(host(xt), ref["x"])
    assert err <= TOL[synth.F32], err
    check_audit(audit.cpu().numpy(), ref["audit"], synth.F32)


def test_guided_with_cond_cache_matches_oracle():
    """Classifier-free guidance: the B model rows carry the conditional and unconditional
    vectors, each with its own c_t."""
    need_gpu()
    cfg = synth.get_config("tiny", B=4, cfg_pairs=1, cfg_scale=3.0)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    against_oracle(cfg, W, inp, abi.FF_FEATFIX, synth.site_mask(cfg), label="guided: ")


def test_cond_cache_refusals_on_gpu():
    """After step 0 the cache cannot be enabled, and a later step must pass step 0's cond."""
    need_gpu()
    cfg = synth.get_config("tiny")
    W = synth.make_weights(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    r = pipeline.Runner(dm, abi.FF_FEATFIX, synth.site_mask(cfg), cond_cache=True)
    x, c, _ = pipeline.host_inputs_to_device(cfg, synth.make_inputs(cfg))
    xs, a = r.start(x)
    r.step(0, xs, c)
    with pytest.raises(abi.FFError) as e:
        r.step(1, xs, c.clone())
    assert e.value.status == abi.FF_E_STATE
    with pytest.raises(abi.FFError) as e:
        abi.ff_ctx_cond_cache(r.ctx, r.ccache.data_ptr(), r.ccache.numel())
    assert e.value.status == abi.FF_E_STATE
    r.step(1, xs, c)   # the same buffer is accepted
    torch.cuda.synchronize()
    r.close()
