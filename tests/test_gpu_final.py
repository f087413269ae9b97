"""The bf16 final layer (LN + modulation + final linear + unpatchify + Euler, Eq. 1's output
head) on MFMA: whole loops against the oracle at shapes that take that kernel (at most 32
outputs per token, C a multiple of 16 up to 1536) with token rows ragged against its
8-row workgroups, k steps that do not split evenly over its eight wavefronts, 8, 24 and
32 outputs per token, and the widest C it takes."""
import numpy as np
import pytest

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import TOL, check_audit, host, need_gpu, say

pytestmark = pytest.mark.gpu

PLAN_KEYS = ("step_kind", "refresh_ord", "k_eff", "read_slots", "write_slot", "action")

CASES = {
    # 3 x 90 = 270 rows (34 workgroups of 8 rows, the last with 6); C = 240: 15 k steps
    "ragged_c240": dict(C=240, H=5, d=48, mlp=960, lat=(4, 1, 20, 18), n_img=90, B=3),
    # lat_c = 8: 32 outputs per token
    "p32": dict(C=256, H=4, d=64, mlp=1024, lat=(8, 1, 16, 16), n_img=64, B=2),
    # the widest C (96 k steps, 12 per wavefront), 48 rows
    "c1536": dict(C=1536, H=12, d=128, mlp=3072, lat=(4, 1, 8, 8), n_img=16, B=3),
    # 8 and 24 outputs per token: weight rows masked inside the MFMA's 32 output columns
    "p8": dict(C=256, H=4, d=64, mlp=1024, lat=(2, 1, 16, 16), n_img=64, B=2),
    "p24": dict(C=256, H=4, d=64, mlp=1024, lat=(6, 1, 12, 12), n_img=36, B=3),
}


@pytest.mark.parametrize("case", list(CASES))
def test_bf16_final_layer_loop_matches_oracle(case):
    need_gpu()
    cfg = synth.get_config("tiny", dtype=synth.BF16, T=6, **CASES[case])
    d = synth.derived(cfg)
    assert d["P"] <= 32 and cfg["C"] % 16 == 0 and cfg["C"] <= 1536
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    r = pipeline.Runner(dm, abi.FF_FEATFIX, mask)
    x, c, txt = pipeline.host_inputs_to_device(cfg, inp)
    xt, audit, counts = r.run(x, c, txt)
    plan = r.export_plan()
    r.close()
    ref = O.run(cfg, O.FEATFIX, inp, W, mask)
    err = O.max_rel_err(host(xt), ref["x"])
    say(f"final layer {case}: rows {cfg['B'] * cfg['n_img']} C {cfg['C']} P {d['P']}: max rel err {err:.3e}")
    assert err <= TOL[synth.BF16], err
    assert counts == ref["counts"]
    for key in PLAN_KEYS:
        np.testing.assert_array_equal(plan[key], ref["plan"][key])
    check_audit(audit.cpu().numpy(), ref["audit"], synth.BF16, label=f"{case}: ")
