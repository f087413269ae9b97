"""Whole-loop parity of the MMDiT workloads at full width and token count (Eq. 1-5 on the
FLUX-like shape of Table 1 and the Qwen-Image-like and HunyuanVideo-like shapes of
Tables 3-4): reduced-depth stacks (synth.reduced_stack) run through ff_denoise_step in
FeatFix mode, with history sums and the conditioning cache (the benchmarked path) and
layer by layer with per-step conditioning, against the
oracle's results stored by tests/golden/make_mmdit_golden.py (the fp64 oracle needs
20-60 minutes per stack on the host)."""
import json
import os

import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import TOL, check_audit, host, need_gpu, say

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
PLAN_KEYS = ("step_kind", "refresh_ord", "k_eff", "read_slots", "write_slot", "action")
COUNT_KEYS = ("n_full_refresh", "n_paid_checks", "n_forwarded", "n_recomputed")
# the stored latent is float16: |stored - x_T| <= 2^-11 max|x_T|, taken off the bound
F16_STORAGE = 2.0 ** -11


def load(name):
    z = np.load(os.path.join(GOLDEN, f"mmdit_{name}_featfix.npz"), allow_pickle=False)
    out = {k: z[k] for k in z.files}
    out["meta"] = json.loads(str(out["meta"]))
    return out


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["flux", "qwen", "hunyuan"])
def test_full_width_mmdit_loop_matches_oracle(name):
    need_gpu()
    g = load(name)
    cfg = synth.reduced_stack(name)
    assert json.loads(json.dumps(cfg)) == g["meta"]["workload"]
    say(f"{name}: full-width stack of {len(cfg['kinds'])} blocks, {cfg['n_img']} + {cfg['n_txt']} tokens, "
        f"T={cfg['T']} R={cfg['R']} K={cfg['K']} sites {cfg['sites']}; generating weights ...")
    W = synth.make_weights(cfg, **g["meta"]["weights"])
    inp = synth.make_inputs(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    del W
    mask = synth.site_mask(cfg)
    dev_inp = pipeline.host_inputs_to_device(cfg, inp)
    T, L = cfg["T"], len(cfg["kinds"])
    audit_ref = {(i, l): g["audit"][i, l] for i in range(T) for l in range(L) if np.isfinite(g["audit"][i, l]).all()}
    counts_ref = dict(zip(COUNT_KEYS, (int(v) for v in g["counts"])))
    ref_x = g["x"].astype(np.float64)
    # the benchmarked path (history sums and the conditioning cache), and layer by layer
    # with the conditioning formed at every step
    for hist_sums in (True, False):
        r = pipeline.Runner(dm, abi.FF_FEATFIX, mask, hist_sums=hist_sums, cond_cache=hist_sums)
        assert (r.hsum is not None) == hist_sums
        x, audit, counts = r.run(*dev_inp)
        torch.cuda.synchronize()
        plan = r.export_plan()
        r.close()
        xg = host(x)
        err = float(np.abs(xg - ref_x).max() / g["x_absmax"])
        say(f"  {name} hist_sums={hist_sums}: max rel err {err:.3e} (bound {TOL[synth.BF16] - F16_STORAGE:.4e}), "
            f"counts {counts}")
        assert err <= TOL[synth.BF16] - F16_STORAGE, err
        assert counts == counts_ref
        for k in PLAN_KEYS:
            np.testing.assert_array_equal(plan[k], g[k])
        a = audit.cpu().numpy()
        check_audit(a, audit_ref, synth.BF16, label=f"{name} sums={hist_sums} ")
        assert np.isnan(a[~np.isfinite(g["audit"])]).all()
    del dm
    torch.cuda.empty_cache()
