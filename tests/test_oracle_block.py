"""Pins for the oracle's exact blocks (Eq. 1 with the DiT / MMDiT block readings):
a second writing from torch.nn.functional library routines, exact special cases,
and symmetry properties that a mis-indexed implementation breaks."""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

import oracle as O
import synth


def _t(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


def small_cfg(kind, n_txt=0, C=64, H=4, mlp=96, N=11, B=2):
    d = C // H
    return dict(kinds=[kind], C=C, H=H, d=d, mlp=mlp, n_img=N - n_txt, n_txt=n_txt, B=B,
                dtype=synth.F32, ln_eps=1e-6, rel_eps=1e-8, lat=(1, 1, 1, 1), patch=(1, 1, 1))


def perturbed(cfg, layer=0, seed=0):
    W = synth.make_layer_weights(cfg, layer, seed=seed, bias_std=0.05, gain_std=0.2)
    # bigger modulation so the gates are O(1) and every branch matters
    def boost(ws):
        ws = dict(ws)
        ws["mod_w"] = ws["mod_w"] * 10
        return ws
    if cfg["kinds"][layer] == synth.MMDIT_DOUBLE:
        return {s: boost(W[s]) for s in ("txt", "img")}
    return boost(W)


def torch_dit_stream(u, mod, W, H, eps, q_g=None, k_g=None):
    """Pre-attention half of a DiT-style stream with torch ops: returns q, k, v [B,H,N,d]."""
    a1, b1, g1, a2, b2, g2 = mod.chunk(6, dim=-1)
    C = u.shape[-1]
    a = Fn.layer_norm(u, (C,), eps=eps) * (1 + b1[:, None]) + a1[:, None]
    qkv = Fn.linear(a, _t(W["qkv_w"]), _t(W["qkv_b"]))
    B, N, _ = u.shape
    q, k, v = [x.view(B, N, H, C // H).transpose(1, 2) for x in qkv.split(C, dim=-1)]
    if q_g is not None:
        q = Fn.rms_norm(q, (C // H,), weight=_t(q_g), eps=eps)
        k = Fn.rms_norm(k, (C // H,), weight=_t(k_g), eps=eps)
    return q, k, v


def torch_dit_post(u, att, mod, W, eps):
    a1, b1, g1, a2, b2, g2 = mod.chunk(6, dim=-1)
    C = u.shape[-1]
    x1 = u + g1[:, None] * Fn.linear(att, _t(W["o_w"]), _t(W["o_b"]))
    m = Fn.layer_norm(x1, (C,), eps=eps) * (1 + b2[:, None]) + a2[:, None]
    y = Fn.gelu(Fn.linear(m, _t(W["fc1_w"]), _t(W["fc1_b"])), approximate="tanh")
    return x1 + g2[:, None] * Fn.linear(y, _t(W["fc2_w"]), _t(W["fc2_b"]))


def _merge(x):
    B, H, N, d = x.shape
    return x.transpose(1, 2).reshape(B, N, H * d)


def test_dit_block_matches_torch_composition():
    cfg = small_cfg(synth.DIT)
    W = perturbed(cfg)
    rng = np.random.default_rng(0)
    u = rng.standard_normal((2, 11, 64))
    cs = O.silu(rng.standard_normal((2, 64)))
    got = O.dit_block(u, cs, W, cfg)
    U = _t(u)
    mod = Fn.linear(_t(cs), _t(W["mod_w"]), _t(W["mod_b"]))
    q, k, v = torch_dit_stream(U, mod, W, 4, 1e-6)
    att = _merge(Fn.scaled_dot_product_attention(q, k, v))
    ref = torch_dit_post(U, att, mod, W, 1e-6).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-11)
    assert np.abs(got - u).max() > 0.1      # the block really does something


def test_double_block_matches_torch_composition():
    cfg = small_cfg(synth.MMDIT_DOUBLE, n_txt=4)
    W = perturbed(cfg)
    rng = np.random.default_rng(1)
    u = rng.standard_normal((2, 11, 64))
    cs = O.silu(rng.standard_normal((2, 64)))
    got = O.double_block(u, cs, W, cfg)
    U = _t(u)
    parts, mods = {}, {}
    seg = {"txt": slice(0, 4), "img": slice(4, 11)}
    for s in ("txt", "img"):
        mods[s] = Fn.linear(_t(cs), _t(W[s]["mod_w"]), _t(W[s]["mod_b"]))
        parts[s] = torch_dit_stream(U[:, seg[s]], mods[s], W[s], 4, 1e-6, W[s]["q_g"], W[s]["k_g"])
    q, k, v = [torch.cat([parts["txt"][i], parts["img"][i]], dim=2) for i in range(3)]
    att = _merge(Fn.scaled_dot_product_attention(q, k, v))
    ref = torch.cat([torch_dit_post(U[:, seg[s]], att[:, seg[s]], mods[s], W[s], 1e-6)
                     for s in ("txt", "img")], dim=1).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-11)


def test_single_block_matches_torch_composition():
    cfg = small_cfg(synth.MMDIT_SINGLE, n_txt=3)
    W = perturbed(cfg)
    rng = np.random.default_rng(2)
    u = rng.standard_normal((2, 11, 64))
    cs = O.silu(rng.standard_normal((2, 64)))
    got = O.single_block(u, cs, W, cfg)
    U = _t(u)
    a_, b_, g_ = Fn.linear(_t(cs), _t(W["mod_w"]), _t(W["mod_b"])).chunk(3, dim=-1)
    a = Fn.layer_norm(U, (64,), eps=1e-6) * (1 + b_[:, None]) + a_[:, None]
    y = Fn.linear(a, _t(W["lin1_w"]), _t(W["lin1_b"]))
    q, k, v, z = y.split([64, 64, 64, 96], dim=-1)
    hv = lambda x: x.view(2, 11, 4, 16).transpose(1, 2)
    q = Fn.rms_norm(hv(q), (16,), weight=_t(W["q_g"]), eps=1e-6)
    k = Fn.rms_norm(hv(k), (16,), weight=_t(W["k_g"]), eps=1e-6)
    att = _merge(Fn.scaled_dot_product_attention(q, k, hv(v)))
    ref = U + g_[:, None] * Fn.linear(torch.cat([att, Fn.gelu(z, approximate="tanh")], -1),
                                      _t(W["lin2_w"]), _t(W["lin2_b"]))
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-10, atol=1e-11)


@pytest.mark.parametrize("kind,n_txt", [(synth.DIT, 0), (synth.MMDIT_DOUBLE, 4), (synth.MMDIT_SINGLE, 4)])
def test_zero_gates_make_the_block_the_identity(kind, n_txt):
    cfg = small_cfg(kind, n_txt=n_txt)
    W = perturbed(cfg)
    sets = [W["txt"], W["img"]] if kind == synth.MMDIT_DOUBLE else [W]
    for ws in sets:
        ws["mod_w"] = np.zeros_like(ws["mod_w"])
        ws["mod_b"] = np.zeros_like(ws["mod_b"])
    u = np.random.default_rng(3).standard_normal((2, 11, 64))
    cs = np.ones((2, 64))
    np.testing.assert_array_equal(O.block(kind, u, cs, W, cfg), u)


@pytest.mark.parametrize("kind", [synth.DIT, synth.MMDIT_SINGLE])
def test_token_permutation_equivariance(kind):
    cfg = small_cfg(kind)
    W = perturbed(cfg)
    rng = np.random.default_rng(4)
    u = rng.standard_normal((2, 11, 64))
    cs = O.silu(rng.standard_normal((2, 64)))
    perm = rng.permutation(11)
    np.testing.assert_allclose(O.block(kind, u[:, perm], cs, W, cfg),
                               O.block(kind, u, cs, W, cfg)[:, perm], rtol=1e-12, atol=1e-13)


def test_samples_are_independent():
    cfg = small_cfg(synth.DIT)
    W = perturbed(cfg)
    rng = np.random.default_rng(5)
    u = rng.standard_normal((2, 11, 64))
    cs = O.silu(rng.standard_normal((2, 64)))
    both = O.dit_block(u, cs, W, cfg)
    one = O.dit_block(u[1:], cs[1:], W, dict(cfg, B=1))
    np.testing.assert_allclose(both[1:], one, rtol=1e-13, atol=1e-14)


def test_double_block_with_shared_weights_ignores_the_split_point():
    # identical weight sets for both streams: the txt/img split must not matter
    cfg = small_cfg(synth.MMDIT_DOUBLE, n_txt=4)
    W = perturbed(cfg)
    W = {"txt": W["img"], "img": W["img"]}
    rng = np.random.default_rng(6)
    u = rng.standard_normal((2, 11, 64))
    cs = O.silu(rng.standard_normal((2, 64)))
    a = O.double_block(u, cs, W, cfg)
    b = O.double_block(u, cs, W, dict(cfg, n_txt=7, n_img=4))
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("kind,n_txt", [(synth.DIT, 0), (synth.MMDIT_DOUBLE, 4), (synth.MMDIT_SINGLE, 4)])
def test_row_subset_equals_full_block(kind, n_txt):
    cfg = small_cfg(kind, n_txt=n_txt)
    W = perturbed(cfg)
    rng = np.random.default_rng(7)
    u = rng.standard_normal((2, 11, 64))
    cs = O.silu(rng.standard_normal((2, 64)))
    full = O.block(kind, u, cs, W, cfg)
    rows = np.array([0, 3, 4, 10])
    np.testing.assert_allclose(O.block(kind, u, cs, W, cfg, rows=rows), full[:, rows],
                               rtol=1e-13, atol=1e-14)


def test_final_layer_matches_torch_composition():
    cfg = small_cfg(synth.DIT)
    cfg["lat"], cfg["patch"] = (4, 1, 4, 4), (1, 2, 2)
    rng = np.random.default_rng(8)
    G = {"fmod_w": rng.standard_normal((128, 64)) * 0.1, "fmod_b": rng.standard_normal(128) * 0.1,
         "f_w": rng.standard_normal((16, 64)) * 0.1, "f_b": rng.standard_normal(16) * 0.1}
    x = rng.standard_normal((2, 4, 64))
    cs = O.silu(rng.standard_normal((2, 64)))
    a, b = Fn.linear(_t(cs), _t(G["fmod_w"]), _t(G["fmod_b"])).chunk(2, dim=-1)
    ref = Fn.linear(Fn.layer_norm(_t(x), (64,), eps=1e-6) * (1 + b[:, None]) + a[:, None],
                    _t(G["f_w"]), _t(G["f_b"]))
    np.testing.assert_allclose(O.final_layer(x, cs, G, cfg), ref.numpy(), rtol=1e-12, atol=1e-13)


def test_conditioning_matches_torch_composition():
    rng = np.random.default_rng(9)
    G = {"t1_w": rng.standard_normal((32, 256)) * 0.05, "t1_b": rng.standard_normal(32) * 0.1,
         "t2_w": rng.standard_normal((32, 32)) * 0.1, "t2_b": rng.standard_normal(32) * 0.1}
    c = rng.standard_normal((3, 32))
    t = 0.37
    half = 128
    f = torch.exp(-np.log(10000.0) * torch.arange(half, dtype=torch.float64) / half)
    phi = torch.cat([torch.cos(1000 * t * f), torch.sin(1000 * t * f)])
    ref = _t(c) + Fn.linear(Fn.silu(Fn.linear(phi, _t(G["t1_w"]), _t(G["t1_b"]))), _t(G["t2_w"]), _t(G["t2_b"]))
    np.testing.assert_allclose(O.conditioning(c, t, G), ref.numpy(), rtol=1e-12, atol=1e-13)


def test_flux_flop_model_against_table_1():
    # Table 1's Vanilla rows (fixture with its citation): 74.69 / 74.39 TFLOP per step
    import json
    import os
    fx = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "table1_flux_vanilla_tflops.json")))
    cfg = synth.get_config("flux")
    per_step = sum(O.block_flops(cfg, k) for k in cfg["kinds"])
    for row in fx["rows"]:
        paper = row["tflops"] * 1e12 / row["steps"]
        assert abs(per_step / paper - 1) < fx["tolerance_rel"], (row, per_step)


def rope_cfg(kind, n_txt=3, C=64, H=2, axes=(8, 12, 12), theta=10000.0):
    """A block with rotary q / k over a 2 x 3 x 4 patch grid (frames, rows, columns)."""
    d = C // H
    cfg = small_cfg(kind, n_txt=n_txt, C=C, H=H, N=n_txt + 24)
    cfg.update(lat=(4, 2, 6, 8), patch=(1, 2, 2), rope_axes=axes, rope_theta=theta)
    assert sum(axes) == d
    return cfg


def torch_rope(x, cfg):
    """Rotary embedding written as complex multiplication: consecutive dim pairs of each
    head vector are complex numbers, multiplied by exp(i * pos_a * theta^(-2k / d_a)) per
    axis chunk; positions from a meshgrid of the patch grid, text rows at the origin."""
    _, F, Hh, Wd = cfg["lat"]
    pt, ph, pw = cfg["patch"]
    grid = torch.meshgrid(torch.arange(F // pt), torch.arange(Hh // ph), torch.arange(Wd // pw), indexing="ij")
    img = torch.stack([g.reshape(-1) for g in grid], dim=-1).double()
    pos = torch.cat([torch.zeros(cfg["n_txt"], 3, dtype=torch.float64), img], dim=0)     # [N, 3]
    rot = []
    for a, da in enumerate(cfg["rope_axes"]):
        freq = cfg["rope_theta"] ** (-torch.arange(0, da, 2, dtype=torch.float64) / da)
        rot.append(torch.polar(torch.ones(pos.shape[0], da // 2, dtype=torch.float64), pos[:, a:a + 1] * freq))
    rot = torch.cat(rot, dim=-1)                                                        # [N, d/2]
    xc = torch.view_as_complex(x.reshape(*x.shape[:-1], -1, 2).contiguous())
    return torch.view_as_real(xc * rot).reshape(x.shape)


def test_double_block_with_rope_matches_torch_composition():
    """q and k are rotated after their per-head RMS norms, over the joint [txt; img] rows."""
    cfg = rope_cfg(synth.MMDIT_DOUBLE)
    W = perturbed(cfg)
    rng = np.random.default_rng(10)
    N, nt = cfg["n_txt"] + cfg["n_img"], cfg["n_txt"]
    u = rng.standard_normal((2, N, 64))
    cs = O.silu(rng.standard_normal((2, 64)))
    got = O.double_block(u, cs, W, cfg)
    U = _t(u)
    parts, mods = {}, {}
    seg = {"txt": slice(0, nt), "img": slice(nt, N)}
    for s in ("txt", "img"):
        mods[s] = Fn.linear(_t(cs), _t(W[s]["mod_w"]), _t(W[s]["mod_b"]))
        parts[s] = torch_dit_stream(U[:, seg[s]], mods[s], W[s], 2, 1e-6, W[s]["q_g"], W[s]["k_g"])
    q, k, v = [torch.cat([parts["txt"][i], parts["img"][i]], dim=2) for i in range(3)]
    att = _merge(Fn.scaled_dot_product_attention(torch_rope(q, cfg), torch_rope(k, cfg), v))
    ref = torch.cat([torch_dit_post(U[:, seg[s]], att[:, seg[s]], mods[s], W[s], 1e-6)
                     for s in ("txt", "img")], dim=1).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-11)
    # the rotation matters: without it the block differs
    assert np.abs(got - O.double_block(u, cs, W, dict(cfg, rope_axes=(0, 0, 0)))).max() > 1e-3


def test_single_block_with_rope_matches_torch_composition():
    cfg = rope_cfg(synth.MMDIT_SINGLE, axes=(4, 14, 14))
    W = perturbed(cfg)
    rng = np.random.default_rng(11)
    N = cfg["n_txt"] + cfg["n_img"]
    u = rng.standard_normal((2, N, 64))
    cs = O.silu(rng.standard_normal((2, 64)))
    got = O.single_block(u, cs, W, cfg)
    U = _t(u)
    a_, b_, g_ = Fn.linear(_t(cs), _t(W["mod_w"]), _t(W["mod_b"])).chunk(3, dim=-1)
    a = Fn.layer_norm(U, (64,), eps=1e-6) * (1 + b_[:, None]) + a_[:, None]
    y = Fn.linear(a, _t(W["lin1_w"]), _t(W["lin1_b"]))
    q, k, v, z = y.split([64, 64, 64, 96], dim=-1)
    hv = lambda x: x.view(2, N, 2, 32).transpose(1, 2)
    q = torch_rope(Fn.rms_norm(hv(q), (32,), weight=_t(W["q_g"]), eps=1e-6), cfg)
    k = torch_rope(Fn.rms_norm(hv(k), (32,), weight=_t(W["k_g"]), eps=1e-6), cfg)
    att = _merge(Fn.scaled_dot_product_attention(q, k, hv(v)))
    ref = U + g_[:, None] * Fn.linear(torch.cat([att, Fn.gelu(z, approximate="tanh")], -1),
                                      _t(W["lin2_w"]), _t(W["lin2_b"]))
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-10, atol=1e-11)
