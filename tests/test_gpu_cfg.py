"""GPU parity of classifier-free guidance by batch doubling (rows b and B/2 + b are a
conditional / unconditional pair reading latent b; v = v_u + s (v_c - v_u)) through
ff_denoise_step, against the oracle."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import TOL, check_audit, host, need_gpu, say

pytestmark = pytest.mark.gpu


def check(cfg, W, inp, mode, mask, dm=None, fused=False):
    dm = dm or pipeline.DeviceModel.from_host(cfg, *W)
    run = pipeline.Runner(dm, mode, mask, hist_sums=fused, cond_cache=fused)
    assert (run.hsum is not None) == fused and (run.ccache is not None) == fused
    x, c, txt = pipeline.host_inputs_to_device(cfg, inp)
    assert x.shape[0] == cfg["B"] // 2
    xt, audit, counts = run.run(x, c, txt)
    torch.cuda.synchronize()
    run.close()
    ref = O.run(cfg, mode, inp, W, mask)
    tol = TOL[cfg["dtype"]]
    err = O.max_rel_err(host(xt), ref["x"])
    say(f"  guided {cfg['name']} B={cfg['B']} s={cfg['cfg_scale']} mode={mode}: max rel err {err:.3e} (tol {tol})")
    assert err <= tol, err
    assert counts == ref["counts"]
    check_audit(audit.cpu().numpy(), ref["audit"], cfg["dtype"])


@pytest.mark.parametrize("B", [2, 4])
@pytest.mark.parametrize("mode", [abi.FF_FEATFIX, abi.FF_VANILLA, abi.FF_VERIFY])
def test_tiny_fp32_guided_loop(B, mode):
    need_gpu()
    cfg = synth.get_config("tiny", B=B, T=8, cfg_pairs=1, cfg_scale=4.0)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    say(f"guided tiny fp32 B={B} mode={mode}")
    check(cfg, W, synth.make_inputs(cfg), mode, synth.site_mask(cfg))


@pytest.mark.parametrize("B", [16, 20])
def test_tiny_bf16_guided_loop_wide_batch(B):
    # 8 and 10 guided pairs: the modulation GEMVs read the SiLU split in two and three
    # groups of 8 samples
    need_gpu()
    cfg = synth.get_config("tiny", B=B, T=8, dtype=synth.BF16, cfg_pairs=1, cfg_scale=4.0)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    say(f"guided tiny bf16 B={B}")
    check(cfg, W, synth.make_inputs(cfg), abi.FF_FEATFIX, synth.site_mask(cfg))


def test_dit_xl2_reduced_depth_guided_loop():
    """DiT-XL/2 width, tokens and batch 8 (4 guided pairs), 4 blocks, bf16, 6 steps: the
    unfused final layer and the guided Euler step at full size."""
    need_gpu()
    cfg = synth.get_config("dit_xl2", kinds=[synth.DIT] * 4, T=6, sites=[1, 3], cfg_pairs=1, cfg_scale=4.0)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    say("guided dit_xl2 reduced depth")
    check(cfg, W, synth.make_inputs(cfg), abi.FF_FEATFIX, synth.site_mask(cfg))


def test_mmdit_guided_loop_with_text():
    """Double + single blocks with text tokens (each twin has its own text rows), bf16."""
    need_gpu()
    cfg = synth.get_config("flux", kinds=[synth.MMDIT_DOUBLE] * 2 + [synth.MMDIT_SINGLE] * 2, C=256, H=2, d=128,
                           mlp=1024, n_txt=24, lat=(16, 1, 20, 18), n_img=90, T=8, R=3, sites=[1, 3], B=2,
                           cfg_pairs=1, cfg_scale=3.5)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    say("guided mmdit with text")
    check(cfg, W, synth.make_inputs(cfg), abi.FF_FEATFIX, synth.site_mask(cfg))


def test_dit_width_guided_loop_benchmarked_path():
    """Guidance on the path the benchmark's guided loop runs: DiT-XL/2 width and tokens,
    2 guided pairs, bf16, K = 2 (step 7 drafts from three refreshes), sites at layers 2
    and 5 of 6 so that runs of two drafted layers come from history sums, and the
    conditioning cache holding both twins' c_t."""
    need_gpu()
    cfg = synth.get_config("dit_xl2", kinds=[synth.DIT] * 6, B=4, T=8, R=3, sites=[2, 5], cfg_pairs=1,
                           cfg_scale=4.0)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    say("guided dit_xl2 width, history sums and conditioning cache")
    check(cfg, W, synth.make_inputs(cfg), abi.FF_FEATFIX, synth.site_mask(cfg), fused=True)
