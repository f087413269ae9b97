"""The bf16 loop refreshes the feature history (Eq. 2: slot <- h - u, rounded to bf16) from
the epilogue of each exact block's last GEMM rather than in a separate pass (or slot <- h
when the history holds block outputs).  At a refresh step every layer is exact, so the
per-layer traces give each layer's input u (the previous layer's output) and output h:
the slot the loop wrote must equal ff_cache_update(u, h) bit for bit.  Shapes are ragged
against the GEMM tiles (rows and columns cut at the ends), for DiT blocks and for MMDiT
double (text, then image stream) and single blocks."""
import numpy as np
import pytest
import torch

import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import need_gpu, say

pytestmark = pytest.mark.gpu

CASES = {
    # 3 x 90 = 270 rows; C = 240: the 96-wide column tiles of the gated GEMMs end half full
    "dit_ragged": lambda: synth.get_config("tiny", kinds=[synth.DIT] * 4, dtype=synth.BF16, C=240, H=5, d=48,
                                           mlp=960, lat=(4, 1, 20, 18), n_img=90, B=3, T=4, R=2),
    # text rows first; C = 256 with 24 + 90 rows per sample
    "mmdit": lambda: synth.get_config("flux", kinds=[synth.MMDIT_DOUBLE] * 2 + [synth.MMDIT_SINGLE] * 2,
                                      C=256, H=2, d=128, mlp=1024, n_txt=24, lat=(16, 1, 20, 18), n_img=90,
                                      B=2, T=4, R=2, sites=[1], dtype=synth.BF16),
}


@pytest.mark.parametrize("feature_mode", [abi.FF_RESIDUAL, abi.FF_OUTPUT])
@pytest.mark.parametrize("case", list(CASES))
def test_fused_refresh_equals_cache_update(case, feature_mode):
    need_gpu()
    cfg = CASES[case]()
    assert cfg["dtype"] == synth.BF16
    L, B, N, C = len(cfg["kinds"]), cfg["B"], cfg["n_img"] + cfg["n_txt"], cfg["C"]
    E = B * N * C
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    dm = pipeline.DeviceModel.from_host(cfg, *W)
    r = pipeline.Runner(dm, abi.FF_FEATFIX, synth.site_mask(cfg), feature_mode=feature_mode)
    trace = torch.empty(L * E, dtype=torch.bfloat16, device="cuda")
    r.trace_into(trace)
    x0, c, txt = pipeline.host_inputs_to_device(cfg, inp)
    x, _ = r.start(x0, audit=False)
    r.step(0, x, c, txt)   # step 0 is a refresh: every layer exact, every layer's slot written
    slot = int(r.export_plan()["write_slot"][0])
    ref = torch.zeros_like(r.cache)
    s = torch.cuda.current_stream().cuda_stream
    for l in range(1, L):
        u = trace[(l - 1) * E:].data_ptr() if feature_mode == abi.FF_RESIDUAL else None
        abi.ff_cache_update(dm.desc, ref.data_ptr(), r.S, l, slot, u, trace[l * E:].data_ptr(), feature_mode, s)
    torch.cuda.synchronize()
    got = r.cache.view(torch.int16)[: L * r.S * E].view(L, r.S, E)
    exp = ref.view(torch.int16)[: L * r.S * E].view(L, r.S, E)
    r.close()
    for l in range(1, L):
        g, e = got[l, slot].cpu().numpy(), exp[l, slot].cpu().numpy()
        nbad = int(np.count_nonzero(g != e))
        say(f"fused refresh {case} mode {feature_mode} layer {l} ({cfg['kinds'][l]}): {E} values, {nbad} differ")
        assert nbad == 0, f"{case}: layer {l}: {nbad} of {E} history values differ from ff_cache_update"
        assert np.count_nonzero(e) > E // 2   # the slot holds data, not a cleared buffer
