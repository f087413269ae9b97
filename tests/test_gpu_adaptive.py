"""GPU runs of the adaptive (discrepancy-triggered) refresh policy through
ff_denoise_step: bitwise against the fixed schedules it reduces to, and against the
oracle's decisions and latent at a threshold chosen from the oracle's own
discrepancies, away from every value that decides a step."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import TOL, host, need_gpu, say

pytestmark = pytest.mark.gpu


def gpu_run(cfg, W, inp, mode, mask, tau, R=None, dm=None):
    dm = dm or pipeline.DeviceModel.from_host(cfg, *W)
    run = pipeline.Runner(dm, mode, mask, R=R, tau=tau)
    x, c, txt = pipeline.host_inputs_to_device(cfg, inp)
    xt, audit, counts = run.run(x, c, txt)
    torch.cuda.synchronize()
    kinds = run.step_kinds()
    run.close()
    return host(xt), audit, counts, kinds


def tiny(T=9, R=3, dtype=synth.F32):
    cfg = dict(synth.get_config("tiny", dtype=dtype))
    cfg["T"], cfg["R"] = T, R
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    return cfg, W, synth.make_inputs(cfg)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_adaptive_limits_are_fixed_schedules_bitwise(dtype):
    need_gpu()
    cfg, W, inp = tiny(dtype=dtype)
    mask = synth.site_mask(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    say(f"adaptive limits dtype={dtype}")
    fixed = gpu_run(cfg, W, inp, abi.FF_FEATFIX, mask, 0.0, dm=dm)
    huge = gpu_run(cfg, W, inp, abi.FF_FEATFIX, mask, 1e30, dm=dm)
    assert np.array_equal(huge[0], fixed[0]) and huge[2] == fixed[2]
    assert list(huge[3]) == [abi.FF_STEP_REFRESH if i % 3 == 0 else abi.FF_STEP_CACHED for i in range(9)]
    # every cached step is checked and every discrepancy exceeds 1e-30: refresh, check,
    # refresh, ... which is the fixed schedule with R = 2
    small = gpu_run(cfg, W, inp, abi.FF_FEATFIX, mask, 1e-30, dm=dm)
    fixed2 = gpu_run(cfg, W, inp, abi.FF_FEATFIX, mask, 0.0, R=2, dm=dm)
    assert list(small[3]) == [abi.FF_STEP_REFRESH if i % 2 == 0 else abi.FF_STEP_CACHED for i in range(9)]
    assert np.array_equal(small[0], fixed2[0]) and small[2] == fixed2[2]


def step_maxima(audit, T):
    """Largest discrepancy of each checked step (the value that decides the next step)."""
    out = {}
    for (i, l), d in audit.items():
        out[i] = max(out.get(i, -np.inf), float(np.max(d)))
    return out


def pick_tau(cfg, W, inp, mode, mask, margin=1e-2):
    """A threshold from the oracle alone: between two of the fixed run's step maxima, such
    that the adaptive run triggers some but not all refreshes and no deciding value lies
    within `margin` (relative) of it."""
    fixed = O.run(cfg, mode, inp, W, mask)
    vals = sorted(set(step_maxima(fixed["audit"], cfg["T"]).values()))
    for lo, hi in zip(vals, vals[1:]):
        tau = float(np.sqrt(lo * hi))
        ref = O.run(cfg, mode, inp, W, mask, tau=tau)
        dec = step_maxima(ref["audit"], cfg["T"]).values()
        early = sum(1 for i, k in enumerate(ref["step_kind"]) if k == O.REFRESH_STEP and i % cfg["R"])
        if early and all(abs(d - tau) > margin * tau for d in dec) and ref["step_kind"] != fixed["step_kind"]:
            return tau, ref
    pytest.skip("no threshold with a clear margin for these inputs")


@pytest.mark.parametrize("mode", [abi.FF_FEATFIX, abi.FF_VERIFY])
def test_adaptive_decisions_and_latent_match_oracle(mode):
    need_gpu()
    cfg, W, inp = tiny(T=10, R=4)
    mask = synth.site_mask(cfg)
    omode = O.FEATFIX if mode == abi.FF_FEATFIX else O.VERIFY
    tau, ref = pick_tau(cfg, W, inp, omode, mask)
    say(f"adaptive tiny fp32 mode={mode} tau={tau:.4e} oracle kinds {ref['step_kind']}")
    x, audit, counts, kinds = gpu_run(cfg, W, inp, mode, mask, tau)
    assert list(kinds) == ref["step_kind"]
    assert counts == ref["counts"]
    err = O.max_rel_err(x, ref["x"])
    assert err <= TOL[cfg["dtype"]], err
    a = audit.cpu().numpy()
    for (i, l), d in ref["audit"].items():
        np.testing.assert_allclose(a[i, l], d, rtol=0, atol=TOL[cfg["dtype"]])
