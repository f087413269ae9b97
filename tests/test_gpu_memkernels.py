"""GPU parity of the HBM-bound kernels (history refresh, Taylor draft, verify+replace)
against the oracle's finite-difference recursion, at the small shape and at every
workload's real per-layer tensor size."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import dev, host, need_gpu, say, ulp_close

pytestmark = pytest.mark.gpu

def layer_cfg(name, **over):
    cfg = synth.get_config(name, **over)
    return cfg


def rnd_for(cfg):
    return O.round_bf16 if cfg["dtype"] == synth.BF16 else (lambda a: a)


@pytest.mark.parametrize("name", ["tiny", "dit_xl2", "flux", "hunyuan"])
@pytest.mark.parametrize("feature_mode", [abi.FF_RESIDUAL, abi.FF_OUTPUT])
def test_refresh_draft_verify_match_oracle(name, feature_mode):
    need_gpu()
    cfg = layer_cfg(name)
    B, N, C = cfg["B"], cfg["n_img"] + cfg["n_txt"], cfg["C"]
    E = B * N * C
    say(f"memkernels {name} E={E} feature_mode={feature_mode}")
    T, R, K, S = cfg["T"], cfg["R"], cfg["K"], cfg["S"]
    dt = pipeline.torch_dtype(cfg)
    bf = cfg["dtype"] == synth.BF16
    rnd = rnd_for(cfg)
    m = pipeline.model_desc(cfg)
    ws_bytes = abi.ff_workspace_bytes(m)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    # one layer's cache only (layer index 0 of a view with n_slots S)
    cache = torch.empty(S * E, dtype=dt, device="cuda")
    # plan for the schedule, draft of layer 0 at the cached step two refreshes in (or the last one)
    mask = np.zeros((T, len(cfg["kinds"])), np.uint8)
    p = abi.ff_plan_build(abi.ff_sched_desc(T, R, K, S, 1e-8, abi.FF_FEATFIX, feature_mode), len(cfg["kinds"]), mask)
    plan = abi.ff_plan_export(p, T, len(cfg["kinds"]), K)
    abi.ff_plan_destroy(p)
    i_star = (K + 1) * R + max(1, R // 2)   # a cached step with k_eff = K
    assert i_star < T
    assert plan["step_kind"][i_star] == abi.FF_STEP_CACHED
    j = plan["refresh_ord"][i_star]
    ke = int(plan["k_eff"][i_star])
    slots = [int(s) for s in plan["read_slots"][i_star][:ke + 1]]
    coeffs = [float(c) for c in plan["coeffs"][i_star][:ke + 1]]
    # a smooth synthetic history: Delta_j = a + b tau + c tau^2 + noise, rounded where the GPU stores it
    rng = np.random.default_rng(7)
    base = [synth.normal((E,), 11 + q, std=1.0) for q in range(3)]
    tc = O.TaylorCache(K)
    for jj in range(j + 1):
        tau = jj * R
        u = synth.normal((E,), 100 + jj, bf16=bf)
        delta = base[0] + 0.05 * tau * base[1] + 0.002 * tau * tau * base[2]
        h = rnd(u.astype(np.float64) + delta).astype(np.float32)
        ud, hd_ = dev(u, dt), dev(h, dt)
        abi.ff_cache_update(m, cache.data_ptr(), S, 0, jj % S, ud.data_ptr() if feature_mode == abi.FF_RESIDUAL else None,
                            hd_.data_ptr(), feature_mode)
        tc.refresh(rnd(h.astype(np.float64) - u.astype(np.float64)) if feature_mode == abi.FF_RESIDUAL
                   else h.astype(np.float64), tau)
    torch.cuda.synchronize()
    # the cached slot of the last refresh holds rnd(h - u) exactly
    u_in = synth.normal((E,), 999, bf16=bf)
    F = tc.forecast(i_star)
    ref = rnd(u_in.astype(np.float64) + F) if feature_mode == abi.FF_RESIDUAL else rnd(F)
    ud = dev(u_in, dt)
    out = torch.empty(E, dtype=dt, device="cuda")
    uptr = ud.data_ptr() if feature_mode == abi.FF_RESIDUAL else None
    abi.ff_draft_forecast(m, cache.data_ptr(), S, 0, ke, slots, coeffs, uptr, out.data_ptr())
    torch.cuda.synchronize()
    got = host(out)
    nbad = ulp_close(got, ref, cfg["dtype"])
    say(f"  draft: k_eff={ke} slots={slots} max|d|={np.abs(got - ref).max():.3e} ulp-misses={nbad}")
    assert nbad <= max(2, E // 100000), nbad
    # in-place draft gives the same bits
    # (in FF_OUTPUT mode the draft ignores u: the output overwrites the buffer it was given)
    inplace = ud.clone()
    abi.ff_draft_forecast(m, cache.data_ptr(), S, 0, ke, slots, coeffs, inplace.data_ptr() if uptr else None,
                          inplace.data_ptr())
    torch.cuda.synchronize()
    assert torch.equal(inplace, out)
    # verify + replace
    hf_np = synth.normal((E,), 555, bf16=bf)
    hf = dev(hf_np, dt)
    rel = torch.zeros(B, dtype=torch.float32, device="cuda")
    for fwd in (1, 0):
        hout = ud.clone()   # in place over u, as the step executor does
        abi.ff_verify_replace(m, cache.data_ptr(), S, 0, ke, slots, coeffs, hout.data_ptr() if uptr else None,
                              hf.data_ptr(), hout.data_ptr(), fwd, 1e-8, rel.data_ptr(), ws.data_ptr(), ws_bytes)
        torch.cuda.synchronize()
        if fwd:
            assert torch.equal(hout, hf), "FeatFix must forward h_f bit for bit"
        else:
            assert torch.equal(hout, out), "Verify must forward exactly the draft"
        ref_d = O.rel_l1(ref.reshape(B, -1), hf_np.astype(np.float64).reshape(B, -1), 1e-8)
        got_d = rel.cpu().numpy().astype(np.float64)
        say(f"  verify fwd={fwd}: rel_l1 gpu={got_d} oracle={ref_d}")
        np.testing.assert_allclose(got_d, ref_d, rtol=1e-3)
    # partial forwarding (the token / channel arms): h_f on every third row / channel of
    # each sample, the draft elsewhere, bit for bit
    for fwd in (abi.FF_FWD_TOKENS, abi.FF_FWD_CHANNELS):
        hout = ud.clone()
        abi.ff_verify_replace(m, cache.data_ptr(), S, 0, ke, slots, coeffs, hout.data_ptr() if uptr else None,
                              hf.data_ptr(), hout.data_ptr(), fwd, 1e-8, rel.data_ptr(), ws.data_ptr(), ws_bytes,
                              stride=3)
        torch.cuda.synchronize()
        sel = torch.zeros((B, N, C), dtype=torch.bool, device="cuda")
        if fwd == abi.FF_FWD_TOKENS:
            sel[:, ::3, :] = True
        else:
            sel[:, :, ::3] = True
        assert torch.equal(hout, torch.where(sel.reshape(-1), hf, out)), f"partial forward {fwd}"
        np.testing.assert_allclose(rel.cpu().numpy().astype(np.float64), ref_d, rtol=1e-3)


def test_memkernels_deterministic():
    need_gpu()
    cfg = synth.get_config("dit_xl2")
    E = cfg["B"] * cfg["n_img"] * cfg["C"]
    m = pipeline.model_desc(cfg)
    ws = torch.empty(abi.ff_workspace_bytes(m), dtype=torch.uint8, device="cuda")
    cache = torch.randn(3 * E, device="cuda").to(torch.bfloat16)
    u = torch.randn(E, device="cuda").to(torch.bfloat16)
    hf = torch.randn(E, device="cuda").to(torch.bfloat16)
    outs, rels = [], []
    for _ in range(2):
        o = u.clone()
        r = torch.zeros(8, device="cuda")
        abi.ff_verify_replace(m, cache.data_ptr(), 3, 0, 2, [0, 2, 1], [1.7, -0.9, 0.2], o.data_ptr(), hf.data_ptr(),
                              o.data_ptr(), 0, 1e-8, r.data_ptr(), ws.data_ptr(), ws.numel())
        torch.cuda.synchronize()
        outs.append(o)
        rels.append(r)
    assert torch.equal(outs[0], outs[1]) and torch.equal(rels[0], rels[1])


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
@pytest.mark.parametrize("feature_mode", [abi.FF_RESIDUAL, abi.FF_OUTPUT])
def test_verify_degenerate_samples(dtype, feature_mode):
    """Eq. 4 at its edges, one case per sample of a single call, at k_eff = 0 (Eq. 2 reduces
    to the last refresh alone) on a shape that fills no tile evenly (35 tokens x 40
    channels): h_f equal to the draft (d = 0 exactly), h_f all zero (d = sum|h_d| / eps),
    draft and h_f both zero (0 / eps = 0 exactly), and an ordinary sample.  Both
    verification entry points must agree bit for bit."""
    need_gpu()
    bf = dtype == synth.BF16
    cfg = synth.get_config("tiny", dtype=dtype, C=40, H=5, d=8, mlp=160, lat=(4, 1, 14, 10), n_img=35, B=4)
    B, N, C = cfg["B"], cfg["n_img"], cfg["C"]
    E, S, eps = B * N * C, 2, 1e-3
    say(f"verify degenerate samples dtype={dtype} feature_mode={feature_mode} E={E}")
    m = pipeline.model_desc(cfg)
    dt = pipeline.torch_dtype(cfg)
    store = O.round_bf16 if bf else (lambda a: np.asarray(a, np.float64).astype(np.float32).astype(np.float64))
    slot_np = synth.normal((S, B, N * C), 31, bf16=bf)
    u_np = synth.normal((B, N * C), 32, bf16=bf)
    slot_np[1, 2] = 0.0   # sample 2: the read slot and u are zero, so the draft is zero
    u_np[2] = 0.0
    res = feature_mode == abi.FF_RESIDUAL
    hd_ref = store(slot_np[1].astype(np.float64) + (u_np if res else 0.0))
    hf_np = synth.normal((B, N * C), 33, bf16=bf).astype(np.float64)
    hf_np[0] = hd_ref[0]   # h_f equal to the draft
    hf_np[1] = 0.0         # h_f zero
    hf_np[2] = 0.0         # h_f zero, draft zero
    cache = dev(slot_np.reshape(-1), dt)
    ud = dev(u_np.reshape(-1), dt) if res else None
    hf = dev(hf_np.reshape(-1), dt)
    ws_bytes = abi.ff_workspace_bytes(m)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    hd = torch.empty(E, dtype=dt, device="cuda")
    uptr = ud.data_ptr() if res else None
    abi.ff_draft_forecast(m, cache.data_ptr(), S, 0, 0, [1], [1.0], uptr, hd.data_ptr())
    outs, rels = [], []
    for call in (abi.ff_verify_replace, abi.ff_verify_replace_noalloc):
        hout = torch.full((E,), 7.0, dtype=dt, device="cuda")
        rel = torch.full((B,), -1.0, dtype=torch.float32, device="cuda")
        extra = (ws.data_ptr(), ws_bytes) if call is abi.ff_verify_replace else ()
        call(m, cache.data_ptr(), S, 0, 0, [1], [1.0], uptr, hf.data_ptr(), hout.data_ptr(), abi.FF_FWD_DRAFT, eps,
             rel.data_ptr(), *extra)
        outs.append(hout)
        rels.append(rel)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(hd).reshape(B, -1), hd_ref)   # one rounding of one exact sum
    assert torch.equal(outs[0], hd) and torch.equal(outs[1], hd), "Verify forwards the draft"
    assert torch.equal(rels[0], rels[1]), "both entry points take the same fixed-order sums"
    got = rels[0].cpu().numpy().astype(np.float64)
    ref = O.rel_l1(hd_ref, hf_np, eps)
    say(f"  rel_l1 gpu={got} oracle={ref}")
    assert got[0] == 0.0 and got[2] == 0.0, got
    assert ref[1] > 1e3   # sum|h_d| over eps
    np.testing.assert_allclose(got[[1, 3]], ref[[1, 3]], rtol=1e-4)
