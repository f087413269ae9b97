"""Per-layer feature traces (ff_ctx_trace) and the rel-L1 distance (ff_rel_l1): FeatFix and
Verify runs against a shadow Vanilla run, layer by layer and step by step, checked
against the same distances between the oracle's own traces; tracing leaves the latent
bit for bit unchanged."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import TOL, host, need_gpu, say

pytestmark = pytest.mark.gpu


def traced_distances(cfg, W, inp, mode, mask, dm):
    """GPU: run `mode` and Vanilla in lockstep with traces; d[i, l, b] = rel-L1 of the mode's
    stream after (i, l) against Vanilla's (ff_rel_l1)."""
    T, L, B = cfg["T"], len(cfg["kinds"]), cfg["B"]
    dt = pipeline.torch_dtype(cfg)
    E = B * (cfg["n_img"] + cfg["n_txt"]) * cfg["C"]
    runs = [pipeline.Runner(dm, mode, mask), pipeline.Runner(dm, abi.FF_VANILLA, mask)]
    bufs = [torch.empty(L * E, dtype=dt, device="cuda") for _ in runs]
    xs = []
    x0, c, txt = pipeline.host_inputs_to_device(cfg, inp)
    for r, b in zip(runs, bufs):
        r.trace_into(b)
        x, _ = r.start(x0, audit=False)
        xs.append(x)
    rel = torch.zeros(B, dtype=torch.float32, device="cuda")
    d = np.zeros((T, L, B))
    for i in range(T):
        for r, x in zip(runs, xs):
            r.step(i, x, c, txt)
        for l in range(L):
            abi.ff_rel_l1(dm.desc, bufs[0][l * E:].data_ptr(), bufs[1][l * E:].data_ptr(), 1e-8, rel.data_ptr(),
                          runs[0].ws.data_ptr(), runs[0].ws_bytes)
            d[i, l] = rel.cpu().numpy()
    torch.cuda.synchronize()
    out = host(xs[0])
    for r in runs:
        r.close()
    return d, out


def oracle_distances(cfg, W, inp, mode, mask):
    T, L = cfg["T"], len(cfg["kinds"])
    tr, tv = [], []
    res = O.run(cfg, mode, inp, W, mask, trace=tr)
    O.run(cfg, O.VANILLA, inp, W, mask, trace=tv)
    d = np.array([O.rel_l1(a, b, 1e-8) for a, b in zip(tr, tv)]).reshape(T, L, -1)
    return d, res["x"]


@pytest.mark.parametrize("mode", [abi.FF_FEATFIX, abi.FF_VERIFY])
def test_shadow_vanilla_distances_match_oracle(mode):
    need_gpu()
    cfg = synth.get_config("tiny")
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    omode = O.FEATFIX if mode == abi.FF_FEATFIX else O.VERIFY
    got, x = traced_distances(cfg, W, inp, mode, mask, dm)
    ref, xr = oracle_distances(cfg, W, inp, omode, mask)
    say(f"  shadow vanilla mode={mode}: max d {ref.max():.3e}, max |gpu - oracle| {np.abs(got - ref).max():.3e}")
    assert np.all(got[0] == 0.0) and np.all(ref[0] == 0.0)   # step 0 refreshes in both runs
    np.testing.assert_allclose(got, ref, rtol=1e-3, atol=1e-6)
    # tracing applies drafted runs layer by layer: the latent is unchanged
    run = pipeline.Runner(dm, mode, mask)
    x0, c, txt = pipeline.host_inputs_to_device(cfg, inp)
    plain, _, _ = run.run(x0, c, txt, audit=False)
    torch.cuda.synchronize()
    run.close()
    assert np.array_equal(host(plain), x)
    assert O.max_rel_err(x, xr) <= TOL[cfg["dtype"]]
