"""Launch profiling of a context (ff_ctx_profile / ff_ctx_profile_read): profiling leaves the
latent bit for bit unchanged, and the per-class records equal what the plan implies,
counted here from the oracle's schedule and the block shapes (Eq. 1 GEMMs and attention
per exact block, one patch embedding per step, one verify per paid check)."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import host, need_gpu, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,hist_sums", [(synth.F32, False), (synth.BF16, False), (synth.BF16, True)],
                         ids=["fp32", "bf16", "bf16_hist_sums"])
def test_profile_records_match_the_plan(dtype, hist_sums):
    need_gpu()
    cfg = synth.get_config("tiny", dtype=dtype)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    T, L, B, C, M = cfg["T"], len(cfg["kinds"]), cfg["B"], cfg["C"], cfg["mlp"]
    rows, P = B * cfg["n_img"], synth.derived(cfg)["P"]
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    say(f"profile tiny dtype={dtype} hist_sums={hist_sums}")

    def loop(profile):
        r = pipeline.Runner(dm, abi.FF_FEATFIX, mask, hist_sums=hist_sums, cond_cache=hist_sums)
        if profile:
            abi.ff_ctx_profile(r.ctx, 1)
        x, _, counts = r.run(*pipeline.host_inputs_to_device(cfg, inp))
        stats = abi.ff_ctx_profile_read(r.ctx) if profile else None
        again = abi.ff_ctx_profile_read(r.ctx) if profile else None
        r.close()
        torch.cuda.synchronize()
        return host(x), counts, stats, again

    plain, counts, _, _ = loop(False)
    x, counts_p, st, again = loop(True)
    assert np.array_equal(x, plain), "profiling changed the latent"
    assert counts_p == counts
    # the schedule from the oracle's plan: every layer at refresh steps, the sites elsewhere
    ref = O.run(cfg, O.FEATFIX, inp, W, mask)
    n_exact = ref["counts"]["n_full_refresh"] * L + ref["counts"]["n_paid_checks"]
    block_flops = 2.0 * rows * (3 * C * C + C * C + M * C + C * M)
    attn_flops = 4.0 * B * cfg["n_img"] ** 2 * cfg["H"] * cfg["d"]
    say(f"  {n_exact} exact blocks; records " + ", ".join(f"{k} {v['launches']}" for k, v in st.items()))
    assert st["gemm"]["launches"] == 4 * n_exact + T
    np.testing.assert_allclose(st["gemm"]["flops"], n_exact * block_flops + T * 2.0 * rows * C * P, rtol=1e-12)
    assert st["attn"]["launches"] == n_exact
    np.testing.assert_allclose(st["attn"]["flops"], n_exact * attn_flops, rtol=1e-12)
    assert st["verify"]["launches"] == ref["counts"]["n_paid_checks"]
    assert st["norm"]["launches"] + st["draft"]["launches"] >= 2 * n_exact
    if dtype == synth.F32:   # the fp32 loop refreshes every layer's history in its own pass
        assert st["cache"]["launches"] == ref["counts"]["n_full_refresh"] * L
    elif not hist_sums:      # the bf16 loop writes it from each block's last GEMM epilogue
        assert st["cache"]["launches"] == 0
    for k, v in st.items():
        assert (v["ms"] > 0) == (v["launches"] > 0), (k, v)
    assert all(v["launches"] == 0 and v["ms"] == 0 for v in again.values()), "reading clears the record"
