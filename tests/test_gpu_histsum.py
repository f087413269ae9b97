"""Cached loops whose runs of drafted layers are applied from per-run history sums
(ff_ctx_hist_sums): Eq. 2's draft is linear in the history, so a run moves the stream by
the run's summed forecast.  Checked against the oracle (which drafts layer by layer), and
for the bitwise invariants of the mode definitions (Sec. 3.3)."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import TOL, check_audit, host, need_gpu, say

pytestmark = pytest.mark.gpu

MODES = {"vanilla": abi.FF_VANILLA, "draft": abi.FF_DRAFT, "verify": abi.FF_VERIFY, "featfix": abi.FF_FEATFIX,
         "exact_only": abi.FF_EXACT_ONLY}


def run(dm, mode, mask, inputs, hist_sums=True, tau=0.0, cond_cache=False):
    r = pipeline.Runner(dm, mode, mask, hist_sums=hist_sums, tau=tau, cond_cache=cond_cache)
    used = r.hsum is not None
    x, audit, counts = r.run(*inputs)
    torch.cuda.synchronize()
    plan = r.export_plan()
    r.close()
    return x, audit, counts, plan, used


def tiny6(dtype=synth.F32, K=1, S=2):
    """Six DiT blocks, one site at layer 3: runs (0, 3) and (4, 6) on cached steps."""
    return synth.get_config("tiny", kinds=[synth.DIT] * 6, sites=[3], dtype=dtype, K=K, S=S)


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("K,S,dtype", [(1, 2, synth.F32), (2, 3, synth.F32), (2, 3, synth.BF16)])
def test_tiny_loop_with_history_sums_matches_oracle(mode, K, S, dtype):
    need_gpu()
    cfg = tiny6(dtype=dtype, K=K, S=S)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    x, audit, counts, plan, used = run(dm, MODES[mode], mask, pipeline.host_inputs_to_device(cfg, inp))
    assert used == (mode != "vanilla")
    ref = O.run(cfg, MODES[mode], inp, W, mask)
    err = O.max_rel_err(host(x), ref["x"])
    say(f"tiny6 K={K} dtype={dtype} {mode} with history sums: max rel err {err:.3e}")
    assert err <= TOL[dtype], err
    assert counts == ref["counts"]
    for key in ("step_kind", "refresh_ord", "k_eff", "read_slots", "write_slot", "action"):
        np.testing.assert_array_equal(plan[key], ref["plan"][key])
    check_audit(audit.cpu().numpy(), ref["audit"], dtype)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_history_sums_keep_the_bitwise_invariants(dtype):
    """FeatFix == Exact-only and Verify == Draft bit for bit, all sites == Vanilla, repeat
    runs identical; the first check's audit equal in Verify and FeatFix."""
    need_gpu()
    cfg = tiny6(dtype=dtype, K=2, S=3)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = pipeline.host_inputs_to_device(cfg, synth.make_inputs(cfg))
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    mask = synth.site_mask(cfg)
    ff, ff2, eo, ve, dr = (run(dm, m, mask, inp) for m in (abi.FF_FEATFIX, abi.FF_FEATFIX, abi.FF_EXACT_ONLY,
                                                              abi.FF_VERIFY, abi.FF_DRAFT))
    va = run(dm, abi.FF_VANILLA, mask, inp)
    al = run(dm, abi.FF_FEATFIX, np.ones_like(mask), inp)
    assert ff[4] and eo[4] and ve[4] and dr[4]
    assert torch.equal(ff[0], ff2[0])
    assert torch.equal(ff[0], eo[0]), "FeatFix and Exact-only differ"
    assert torch.equal(ve[0], dr[0]), "Verify and Draft differ"
    assert torch.equal(al[0], va[0]), "all-sites FeatFix differs from Vanilla"
    assert not torch.equal(ff[0], ve[0])
    np.testing.assert_array_equal(ff[1][1, 3].cpu().numpy(), ve[1][1, 3].cpu().numpy())
    # the per-layer path agrees to the rounding of the storage type
    pl = run(dm, abi.FF_FEATFIX, mask, inp, hist_sums=False)
    d = O.max_rel_err(host(ff[0]), host(pl[0]))
    say(f"tiny6 dtype={dtype}: sums vs per-layer drafts max rel diff {d:.3e}")
    assert d <= TOL[dtype]


def test_adaptive_limit_with_history_sums():
    """tau = 1e30 never triggers an extra refresh: the adaptive loop with sums equals the
    fixed loop with sums bit for bit (its runs come from every step's cached row)."""
    need_gpu()
    cfg = tiny6(dtype=synth.BF16, K=2, S=3)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = pipeline.host_inputs_to_device(cfg, synth.make_inputs(cfg))
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    mask = synth.site_mask(cfg)
    for mode in (abi.FF_FEATFIX, abi.FF_VERIFY):
        fixed = run(dm, mode, mask, inp)
        adapt = run(dm, mode, mask, inp, tau=1e30)
        assert adapt[4]
        assert torch.equal(fixed[0], adapt[0])
        assert fixed[2] == adapt[2]


def test_enabling_history_sums_mid_run_is_refused():
    need_gpu()
    cfg = tiny6()
    W = synth.make_weights(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    mask = synth.site_mask(cfg)
    r = pipeline.Runner(dm, abi.FF_FEATFIX, mask)
    nb = abi.ff_hist_sum_bytes(dm.desc, r.plan)
    assert nb > 0
    buf = torch.empty(nb, dtype=torch.uint8, device="cuda")
    x0, c, txt = pipeline.host_inputs_to_device(cfg, synth.make_inputs(cfg))
    x, a = r.start(x0)
    r.step(0, x, c, txt, a)
    torch.cuda.synchronize()
    assert abi.lib().ff_ctx_hist_sums(r.ctx, buf.data_ptr(), nb) == abi.FF_E_STATE
    abi.ff_ctx_reset(r.ctx)
    assert abi.lib().ff_ctx_hist_sums(r.ctx, buf.data_ptr(), nb) == abi.FF_OK
    r.close()


def test_dit_xl2_full_depth_with_history_sums_sampled():
    """The DiT-XL/2 workload at full depth and batch 8 (runs 0-12 and 14-26) over 12 steps:
    refreshes at 0, 5 and 10, so steps 11 drafts at second order (k_eff = 2, three history
    terms, the ring of 3 slots full) -- the draft of 32 of the 40 cached steps of the
    50-step loop.  With history sums and the conditioning cache (the benchmarked path) and
    layer by layer, both against the oracle, which follows samples 0 and 7 (samples never
    interact)."""
    need_gpu()
    cfg = synth.get_config("dit_xl2", T=12)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    dev_inp = pipeline.host_inputs_to_device(cfg, inp)
    sums = run(dm, abi.FF_FEATFIX, mask, dev_inp, cond_cache=True)   # the benchmarked path
    assert sums[4]
    per_layer = run(dm, abi.FF_FEATFIX, mask, dev_inp, hist_sums=False)
    del dm
    assert list(sums[3]["k_eff"]) == [0, 0, 0, 0, 0, 1, 1, 1, 1, 1, 2, 2]
    idx = [0, 7]
    say("dit_xl2 full depth T=12: oracle on samples 0 and 7 ...")
    ref = O.run(synth.get_config("dit_xl2", T=12, B=2), O.FEATFIX, {k: v[idx] for k, v in inp.items()}, W, mask)
    for label, (x, audit, counts, plan, _used) in (("sums", sums), ("per-layer", per_layer)):
        err = O.max_rel_err(host(x)[idx], ref["x"])
        say(f"dit_xl2 full depth T=12 {label}: max rel err {err:.3e}")
        assert err <= TOL[synth.BF16], err
        assert counts == ref["counts"]
        for key in ("step_kind", "refresh_ord", "k_eff", "read_slots", "write_slot", "action"):
            np.testing.assert_array_equal(plan[key], ref["plan"][key])
        check_audit(audit.cpu().numpy(), ref["audit"], synth.BF16, idx, label=f"{label} ")


def test_flux_like_full_size_with_history_sums():
    """FLUX-like at full depth and size (runs 0-17, 19-36, 38-55): the invariants hold bit
    for bit with sums, and the latent agrees with per-layer drafts to bf16 rounding."""
    need_gpu()
    cfg = synth.get_config("flux", T=8)
    mask = synth.site_mask(cfg)
    dm = pipeline.DeviceModel.random(cfg, seed=0)
    g = torch.Generator(device="cuda")
    g.manual_seed(1)
    x0 = torch.randn((1,) + tuple(cfg["lat"]), generator=g, device="cuda")
    cond = torch.randn((1, cfg["C"]), generator=g, device="cuda").bfloat16().float()
    txt = torch.randn((1, cfg["n_txt"], cfg["C"]), generator=g, device="cuda").bfloat16()
    inp = (x0, cond, txt)
    ff = run(dm, abi.FF_FEATFIX, mask, inp)
    eo = run(dm, abi.FF_EXACT_ONLY, mask, inp)
    ve = run(dm, abi.FF_VERIFY, mask, inp)
    dr = run(dm, abi.FF_DRAFT, mask, inp)
    pl = run(dm, abi.FF_FEATFIX, mask, inp, hist_sums=False)
    del dm
    assert ff[4] and dr[4]
    assert torch.equal(ff[0], eo[0]) and torch.equal(ve[0], dr[0])
    d = O.max_rel_err(host(ff[0]), host(pl[0]))
    say(f"flux full size: sums vs per-layer drafts max rel diff {d:.3e}")
    assert d <= TOL[synth.BF16]
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", [abi.FF_FEATFIX, abi.FF_VERIFY])
def test_adaptive_refreshes_with_history_sums_match_oracle(mode):
    """A threshold that makes some cached steps trigger a refresh (chosen from the oracle's
    own discrepancies, every deciding value more than 1 % from it): the sums are re-formed
    at the refreshes the run decides, and the GPU takes the oracle's decisions step for
    step with runs (0, 3) and (4, 6) applied from them."""
    from test_gpu_adaptive import pick_tau
    need_gpu()
    cfg = dict(tiny6(K=2, S=3), T=10, R=4)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    tau, ref = pick_tau(cfg, W, inp, O.FEATFIX if mode == abi.FF_FEATFIX else O.VERIFY, mask)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    r = pipeline.Runner(dm, mode, mask, tau=tau, hist_sums=True)
    assert r.hsum is not None
    x, audit, counts = r.run(*pipeline.host_inputs_to_device(cfg, inp))
    torch.cuda.synchronize()
    kinds = r.step_kinds()
    r.close()
    say(f"adaptive tiny6 with sums mode={mode} tau={tau:.4e}: kinds {list(kinds)}")
    assert list(kinds) == ref["step_kind"]
    assert counts == ref["counts"]
    err = O.max_rel_err(host(x), ref["x"])
    assert err <= TOL[synth.F32], err
    check_audit(audit.cpu().numpy(), ref["audit"], synth.F32)
