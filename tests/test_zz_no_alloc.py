"""ff_verify_replace_noalloc (the verify + replace pass with its partial sums in the
library's own device array instead of a caller workspace) against ff_verify_replace on
the same inputs: h_out and rel_l1 bit for bit, on two calls in a row, the second with a
smaller input (the array keeps the first call's contents).  Plus the host-side refusal of
a batch beyond the array's size (no GPU needed)."""
import numpy as np
import pytest
import torch

import synth
from paper_2607_27842_amd import abi, pipeline

MAXB = abi.FF_NOALLOC_VERIFY_MAX_B


def case(cfg, seed):
    """Random cache (S slots of one layer), incoming u and exact h_f of a [B, N, C] site."""
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    dt = pipeline.torch_dtype(cfg)
    E = cfg["B"] * (cfg["n_img"] + cfg["n_txt"]) * cfg["C"]
    L, S = len(cfg["kinds"]), cfg["S"]
    rnd = lambda n: torch.randn(n, generator=g, device="cuda").to(dt)
    return rnd(L * S * E), rnd(E), rnd(E), E


@pytest.mark.gpu
def test_noalloc_verify_equals_workspace_verify_on_two_calls():
    assert torch.cuda.is_available(), "GPU test run without a GPU"
    abi.lib()
    big = synth.get_config("dit_xl2", B=MAXB)                       # largest batch the array takes
    small = synth.get_config("tiny", dtype=synth.BF16, B=2, K=2, S=3)
    for call, (cfg, fwd, seed) in enumerate(((big, abi.FF_FWD_EXACT, 1), (small, abi.FF_FWD_DRAFT, 2))):
        m = pipeline.model_desc(cfg)
        cache, u, hf, E = case(cfg, seed)
        layer, S, K = len(cfg["kinds"]) - 1, cfg["S"], 2
        slots, coeffs = [2 % S, 1 % S, 0], [1.7, -0.9, 0.2]
        ws_bytes = abi.ff_workspace_bytes(m)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
        ref_out, out = torch.empty_like(u), torch.empty_like(u)
        ref_rel = torch.full((cfg["B"],), float("nan"), device="cuda")
        rel = torch.full((cfg["B"],), float("nan"), device="cuda")
        print(f"call {call}: {cfg['name']} B={cfg['B']} E={E} forward={fwd}", flush=True)
        abi.ff_verify_replace(m, cache.data_ptr(), S, layer, K, slots, coeffs, u.data_ptr(), hf.data_ptr(),
                              ref_out.data_ptr(), fwd, cfg["rel_eps"], ref_rel.data_ptr(), ws.data_ptr(), ws_bytes)
        abi.ff_verify_replace_noalloc(m, cache.data_ptr(), S, layer, K, slots, coeffs, u.data_ptr(), hf.data_ptr(),
                                      out.data_ptr(), fwd, cfg["rel_eps"], rel.data_ptr())
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out)
        assert torch.equal(rel, ref_rel) and torch.isfinite(rel).all() and (rel > 0).all()
        if fwd == abi.FF_FWD_EXACT:
            assert torch.equal(out, hf)
        print(f"  rel_l1 {rel.cpu().numpy()}", flush=True)


def test_noalloc_verify_refuses_a_batch_beyond_its_array():
    cfg = synth.get_config("tiny", dtype=synth.BF16, B=MAXB + 1)
    m = pipeline.model_desc(cfg)
    fake = 1 << 20   # aligned stand-in addresses: the call must fail before any device access
    with pytest.raises(abi.FFError) as e:
        abi.ff_verify_replace_noalloc(m, fake, 2, 0, 1, [1, 0], [1.5, -0.5], fake, fake * 2, fake * 3,
                                      abi.FF_FWD_EXACT, 1e-8, fake * 4)
    assert e.value.status == abi.FF_E_WORKSPACE
    assert "B <=" in abi.ff_last_error()
