"""GPU runs of the matched-compute arms (Sec. 3.3: token- and channel-level partial
forwarding, whole-timestep recomputation) through ff_denoise_step: against the oracle on
the tiny fp32 loop, and bit for bit against the modes they reduce to."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import TOL, check_audit, host, need_gpu, say

pytestmark = pytest.mark.gpu

ARMS = {"tokens": (abi.FF_TOKENS_PARTIAL, O.TOKENS_PARTIAL), "channels": (abi.FF_CHANNELS_PARTIAL, O.CHANNELS_PARTIAL),
        "recompute": (abi.FF_RECOMPUTE, O.RECOMPUTE)}


def gpu_run(cfg, W, inp, mode, mask, stride=2, dm=None):
    dm = dm or pipeline.DeviceModel.from_host(cfg, *W)
    run = pipeline.Runner(dm, mode, mask, part_stride=stride)
    x, c, txt = pipeline.host_inputs_to_device(cfg, inp)
    xt, audit, counts = run.run(x, c, txt)
    torch.cuda.synchronize()
    plan = run.export_plan()
    run.close()
    return xt, audit, counts, plan


@pytest.mark.parametrize("arm", list(ARMS))
def test_arm_loops_match_oracle(arm):
    need_gpu()
    cfg = synth.get_config("tiny")
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    gmode, omode = ARMS[arm]
    xt, audit, counts, plan = gpu_run(cfg, W, inp, gmode, mask, stride=3)
    ref = O.run(cfg, omode, inp, W, mask, stride=3)
    err = O.max_rel_err(host(xt), ref["x"])
    say(f"  tiny arm={arm}: max rel err {err:.3e} counts {counts}")
    assert err <= TOL[cfg["dtype"]], err
    assert counts == ref["counts"]
    for key in ("step_kind", "refresh_ord", "k_eff", "read_slots", "write_slot", "action"):
        np.testing.assert_array_equal(plan[key], ref["plan"][key])
    check_audit(audit.cpu().numpy(), ref["audit"], cfg["dtype"])


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_arm_reductions_bitwise(dtype):
    """Stride-1 partial arms == FeatFix; recompute from layer 0 == Vanilla; recompute with
    last-layer sites == FeatFix."""
    need_gpu()
    cfg = synth.get_config("tiny", dtype=dtype)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    T, L = cfg["T"], len(cfg["kinds"])
    mask = synth.site_mask(cfg)
    say(f"arm reductions dtype={dtype}")
    ff = gpu_run(cfg, W, inp, abi.FF_FEATFIX, mask, dm=dm)
    for mode in (abi.FF_TOKENS_PARTIAL, abi.FF_CHANNELS_PARTIAL):
        arm = gpu_run(cfg, W, inp, mode, mask, stride=1, dm=dm)
        assert torch.equal(arm[0], ff[0]), f"stride-1 arm {mode} differs from FeatFix"
        half = gpu_run(cfg, W, inp, mode, mask, stride=2, dm=dm)
        assert not torch.equal(half[0], ff[0])
    first = np.zeros((T, L), np.uint8)
    first[:, 0] = 1
    rc = gpu_run(cfg, W, inp, abi.FF_RECOMPUTE, first, dm=dm)
    va = gpu_run(cfg, W, inp, abi.FF_VANILLA, first, dm=dm)
    assert torch.equal(rc[0], va[0]), "recompute from layer 0 differs from Vanilla"
    last = np.zeros((T, L), np.uint8)
    last[:, L - 1] = 1
    rc = gpu_run(cfg, W, inp, abi.FF_RECOMPUTE, last, dm=dm)
    ffl = gpu_run(cfg, W, inp, abi.FF_FEATFIX, last, dm=dm)
    assert torch.equal(rc[0], ffl[0]), "recompute with last-layer sites differs from FeatFix"


@pytest.mark.parametrize("arm", list(ARMS))
def test_arm_loops_dit_width_benchmarked_path(arm):
    """The arms as the benchmark times them: bf16 at DiT-XL/2 width (C = 1152, 16 heads of
    72, 256 tokens), batch 2, K = 2 (step 7 drafts from three refreshes), sites at layers
    2 and 5 of 6, so that runs of two drafted layers come from history sums, with the
    conditioning cache; against the oracle's latent, plan, counters and audit."""
    need_gpu()
    cfg = synth.get_config("dit_xl2", kinds=[synth.DIT] * 6, sites=[2, 5], B=2, T=8, R=3)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    gmode, omode = ARMS[arm]
    ref = O.run(cfg, omode, inp, W, mask, stride=3)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    run = pipeline.Runner(dm, gmode, mask, part_stride=3, hist_sums=True, cond_cache=True)
    assert run.hsum is not None
    xt, audit, counts = run.run(*pipeline.host_inputs_to_device(cfg, inp))
    torch.cuda.synchronize()
    plan = run.export_plan()
    run.close()
    err = O.max_rel_err(host(xt), ref["x"])
    say(f"  DiT-width bf16 arm={arm} (history sums, conditioning cache): max rel err {err:.3e} counts {counts}")
    assert int(np.max(plan["k_eff"])) == 2
    assert err <= TOL[cfg["dtype"]], err
    assert counts == ref["counts"]
    for key in ("step_kind", "refresh_ord", "k_eff", "read_slots", "write_slot", "action"):
        np.testing.assert_array_equal(plan[key], ref["plan"][key])
    check_audit(audit.cpu().numpy(), ref["audit"], cfg["dtype"])
