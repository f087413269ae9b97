"""Whole cached loops at the full depth and size of the large workloads (FLUX-like,
Qwen-like, HunyuanVideo-like, DiT-XL/2), in the launch configuration the throughput runs
use, checked through properties that hold at any size (the oracle cannot run these loops
in test time): FeatFix equals Exact-only and Verify equals Draft bit for bit (Eq. 5 and the
mode definitions of Sec. 3.3), FeatFix with a site at every layer equals Vanilla, repeated
runs are bitwise identical, and the plan and counters equal the oracle's schedule."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import need_gpu, say

pytestmark = pytest.mark.gpu


def device_inputs(cfg, seed=1):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    c_lat, F, H, W = cfg["lat"]
    dt = pipeline.torch_dtype(cfg)
    x0 = torch.randn((cfg["B"], c_lat, F, H, W), generator=g, device="cuda", dtype=torch.float32)
    cond = torch.randn((cfg["B"], cfg["C"]), generator=g, device="cuda").to(dt).float()
    txt = None
    if cfg["n_txt"] > 0:
        txt = torch.randn((cfg["B"], cfg["n_txt"], cfg["C"]), generator=g, device="cuda").to(dt)
    return x0, cond, txt


def run_loop(dm, mode, mask, inputs):
    r = pipeline.Runner(dm, mode, mask)
    x, audit, counts = r.run(*inputs)
    torch.cuda.synchronize()
    plan = r.export_plan()
    r.close()
    return x, audit, counts, plan


@pytest.mark.parametrize("name", ["flux", "qwen", "hunyuan", "dit_xl2"])
def test_full_size_loop_invariants(name):
    need_gpu()
    base = synth.get_config(name)
    cfg = synth.get_config(name, T=base["R"] + 2)      # two refreshes, R - 1 + 1 cached steps
    L = len(cfg["kinds"])
    mask = synth.site_mask(cfg)
    say(f"{name}: {L} blocks, C={cfg['C']}, tokens {cfg['n_img']}+{cfg['n_txt']}, B={cfg['B']}, "
        f"T={cfg['T']}, R={cfg['R']}, K={cfg['K']}, sites {synth.sites_of(cfg)}")
    dm = pipeline.DeviceModel.random(cfg, seed=0)
    inputs = device_inputs(cfg)
    try:
        ff = run_loop(dm, abi.FF_FEATFIX, mask, inputs)
        ff2 = run_loop(dm, abi.FF_FEATFIX, mask, inputs)
        eo = run_loop(dm, abi.FF_EXACT_ONLY, mask, inputs)
        ve = run_loop(dm, abi.FF_VERIFY, mask, inputs)
        dr = run_loop(dm, abi.FF_DRAFT, mask, inputs)
        va = run_loop(dm, abi.FF_VANILLA, mask, inputs)
        al = run_loop(dm, abi.FF_FEATFIX, np.ones_like(mask), inputs)
    finally:
        del dm
    for label, r in (("featfix", ff), ("verify", ve), ("vanilla", va)):
        assert torch.isfinite(r[0]).all(), f"{label}: non-finite latent"
    assert torch.equal(ff[0], ff2[0]), "repeated FeatFix runs differ"
    assert torch.equal(ff[0], eo[0]), "FeatFix and Exact-only differ"
    assert torch.equal(ve[0], dr[0]), "Verify and Draft differ"
    assert torch.equal(al[0], va[0]), "FeatFix with every layer a site differs from Vanilla"
    assert not torch.equal(ff[0], ve[0]), "forwarding changed nothing"
    assert not torch.equal(ff[0], va[0]), "the cached loop equals Vanilla"
    say(f"  max |FeatFix - Vanilla| {(ff[0] - va[0]).abs().max().item():.4e}, "
        f"max |Verify - Vanilla| {(ve[0] - va[0]).abs().max().item():.4e}")
    for mode, r in ((abi.FF_FEATFIX, ff), (abi.FF_VERIFY, ve), (abi.FF_DRAFT, dr), (abi.FF_VANILLA, va)):
        ref = O.make_plan(cfg["T"], L, cfg["R"], cfg["K"], cfg["S"], mask, mode)
        for key in ("step_kind", "refresh_ord", "k_eff", "read_slots", "write_slot", "action"):
            np.testing.assert_array_equal(r[3][key], ref[key], err_msg=f"mode {mode} {key}")
        assert r[2] == ref["counts"], (mode, r[2], ref["counts"])
    # the audit holds Eq. 4 at the paid sites only, and the first one sees the same
    # incoming state in Verify and FeatFix
    paid = O.make_plan(cfg["T"], L, cfg["R"], cfg["K"], cfg["S"], mask, abi.FF_FEATFIX)["action"] == O.SITE
    for r in (ff, ve):
        a = r[1].cpu().numpy()
        assert np.isfinite(a[paid]).all() and (a[paid] >= 0).all()
        assert np.isnan(a[~paid]).all()
    i0, l0 = np.argwhere(paid)[0]
    np.testing.assert_array_equal(ff[1][i0, l0].cpu().numpy(), ve[1][i0, l0].cpu().numpy())
    torch.cuda.empty_cache()
