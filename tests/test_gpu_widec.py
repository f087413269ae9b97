"""The widest hidden size the LayerNorm kernels take (C = 4096: eight 8-element units per
lane), in a bf16 FeatFix loop with history sums at second order (Eq. 2, K = 2) against the
oracle: the exact blocks' LayerNorms at C = 4096, the run of drafted layers in front of
the site applied by the site block's first LayerNorm (its history terms in two-unit
batches), the verify pass (Eq. 3-5), and the unfused final layer (C above the MFMA final
layer's limit)."""
import numpy as np

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import TOL, check_audit, host, need_gpu, say

import pytest

pytestmark = pytest.mark.gpu


def test_c4096_loop_with_history_sums_matches_oracle():
    need_gpu()
    # three DiT blocks, the site at the last: on cached steps layers 0-1 are a run that the
    # site block's first LayerNorm applies; refreshes at 0, 3, 6 give k_eff = 2 at step 7
    cfg = synth.get_config("tiny", kinds=[synth.DIT] * 3, sites=[2], dtype=synth.BF16, C=4096, H=32, d=128,
                           mlp=4096, lat=(4, 1, 8, 8), n_img=16, B=2, T=8, R=3, K=2, S=3)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    r = pipeline.Runner(dm, abi.FF_FEATFIX, mask, hist_sums=True)
    assert r.hsum is not None
    x, audit, counts = r.run(*pipeline.host_inputs_to_device(cfg, inp))
    plan = r.export_plan()
    r.close()
    ref = O.run(cfg, O.FEATFIX, inp, W, mask)
    err = O.max_rel_err(host(x), ref["x"])
    say(f"C=4096 FeatFix with history sums: k_eff max {int(np.max(plan['k_eff']))}, max rel err {err:.3e}")
    assert int(np.max(plan["k_eff"])) == 2
    assert err <= TOL[synth.BF16], err
    assert counts == ref["counts"]
    for key in ("step_kind", "refresh_ord", "k_eff", "read_slots", "write_slot", "action"):
        np.testing.assert_array_equal(plan[key], ref["plan"][key])
    check_audit(audit.cpu().numpy(), ref["audit"], synth.BF16)
