"""The stored oracle results (tests/golden/*.npz) belong to the current oracle and
workload definitions: written by tests/golden/make_mmdit_golden.py from the oracle source
whose sha256 they record, for the workload synth.reduced_stack describes now; their plan
arrays and counts are the oracle's schedule for that workload."""
import hashlib
import json
import os

import numpy as np
import pytest

import oracle as O
import synth

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PLAN_KEYS = ("step_kind", "refresh_ord", "k_eff", "read_slots", "write_slot", "action")


@pytest.mark.parametrize("name", ["flux", "qwen", "hunyuan"])
def test_golden_file_is_current(name):
    z = np.load(os.path.join(HERE, "golden", f"mmdit_{name}_featfix.npz"), allow_pickle=False)
    meta = json.loads(str(z["meta"]))
    sha = hashlib.sha256(open(os.path.join(ROOT, "oracle", "featfix_oracle.py"), "rb").read()).hexdigest()
    assert meta["oracle_sha256"] == sha, "oracle changed since the golden file was written: rerun make_mmdit_golden.py"
    cfg = synth.reduced_stack(name)
    assert json.loads(json.dumps(cfg)) == meta["workload"]
    T, L = cfg["T"], len(cfg["kinds"])
    plan = O.make_plan(T, L, cfg["R"], cfg["K"], cfg["S"], synth.site_mask(cfg), O.FEATFIX)
    for k in PLAN_KEYS:
        np.testing.assert_array_equal(z[k], plan[k])
    assert [int(v) for v in z["counts"]] == [plan["counts"][k] for k in
                                             ("n_full_refresh", "n_paid_checks", "n_forwarded", "n_recomputed")]
    # an audit entry exactly where a paid check ran, finite and positive
    paid = plan["action"] == O.SITE
    assert np.isfinite(z["audit"][paid]).all() and (z["audit"][paid] > 0).all()
    assert np.isnan(z["audit"][~paid]).all()
    assert z["x"].shape == (cfg["B"],) + tuple(cfg["lat"]) and np.isfinite(z["x"]).all()
    assert abs(float(np.abs(z["x"]).max()) / float(z["x_absmax"]) - 1) < 2.0 ** -10
