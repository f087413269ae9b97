"""Pins for the oracle's primitives against library routines, brute force and closed forms."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

import oracle as O
import synth


def _t(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


def test_round_bf16_matches_torch_on_fp32_values():
    rng = np.random.default_rng(0)
    a = (rng.standard_normal(200000) * np.exp(rng.uniform(-30, 30, 200000))).astype(np.float32)
    # exact ties: bf16 value + half an ulp
    base = torch.randn(1000).to(torch.bfloat16).float().numpy()
    ulp = np.abs(base) * 2.0 ** -7
    ties = (base + ulp / 2).astype(np.float32)
    a = np.concatenate([a, ties, base, [0.0, -0.0, 1e-40, -3e-39]]).astype(np.float32)
    ref = torch.from_numpy(a).to(torch.bfloat16).double().numpy()
    got = O.round_bf16(a.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_round_bf16_is_direct_not_double_rounding():
    # 1 + 2^-8 + 2^-30: nearest bf16 is 1 + 2^-7; rounding through fp32 first would give a tie
    # (1 + 2^-8) that then rounds to even (1.0).
    x = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert O.round_bf16(np.array([x]))[0] == 1.0 + 2.0 ** -7
    assert O.round_bf16(np.array([1.0 + 2.0 ** -8]))[0] == 1.0          # tie -> even
    assert O.round_bf16(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6   # tie -> even (up)
    assert np.isinf(O.round_bf16(np.array([3.4e38]))[0])


def test_synth_bf16_rounding_agrees_with_torch():
    a = np.random.default_rng(1).standard_normal(100000).astype(np.float32)
    np.testing.assert_array_equal(synth.to_bf16_values(a),
                                  torch.from_numpy(a).to(torch.bfloat16).float().numpy())


def test_activations_match_torch():
    z = np.linspace(-12, 12, 2001)
    np.testing.assert_allclose(O.silu(z), Fn.silu(_t(z)).numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(O.gelu_tanh(z), Fn.gelu(_t(z), approximate="tanh").numpy(),
                               rtol=1e-14, atol=1e-15)


def test_layer_norm_and_rms_norm_match_torch():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 7, 96)) * 3 + 1.5
    np.testing.assert_allclose(O.layer_norm(x, 1e-6), Fn.layer_norm(_t(x), (96,), eps=1e-6).numpy(),
                               rtol=1e-12, atol=1e-12)
    g = rng.standard_normal(96)
    np.testing.assert_allclose(O.rms_norm(x, g, 1e-6),
                               Fn.rms_norm(_t(x), (96,), weight=_t(g), eps=1e-6).numpy(),
                               rtol=1e-12, atol=1e-12)


def _attention_brute(q, k, v):
    B, H, Nq, d = q.shape
    N = k.shape[2]
    out = np.zeros((B, H, Nq, v.shape[-1]))
    for b in range(B):
        for h in range(H):
            for i in range(Nq):
                s = [sum(q[b, h, i, e] * k[b, h, j, e] for e in range(d)) / math.sqrt(d)
                     for j in range(N)]
                mx = max(s)
                w = [math.exp(x - mx) for x in s]
                z = sum(w)
                for e in range(v.shape[-1]):
                    out[b, h, i, e] = sum(w[j] * v[b, h, j, e] for j in range(N)) / z
    return out


@pytest.mark.parametrize("N,d", [(1, 8), (5, 8), (17, 8), (5, 72), (17, 72)])
def test_attention_brute_force(N, d):
    rng = np.random.default_rng(N * 100 + d)
    q, k, v = (rng.standard_normal((1, 2, N, d)) for _ in range(3))
    np.testing.assert_allclose(O.attention(q, k, v), _attention_brute(q, k, v), rtol=1e-11, atol=1e-12)


def test_attention_matches_torch_sdpa_and_special_cases():
    rng = np.random.default_rng(3)
    q, k, v = (rng.standard_normal((2, 3, 33, 16)) for _ in range(3))
    ref = Fn.scaled_dot_product_attention(_t(q), _t(k), _t(v)).numpy()
    np.testing.assert_allclose(O.attention(q, k, v), ref, rtol=1e-11, atol=1e-12)
    # one key: output is that value row
    np.testing.assert_allclose(O.attention(q[:, :, :4], k[:, :, :1], v[:, :, :1]),
                               np.broadcast_to(v[:, :, :1], (2, 3, 4, 16)), rtol=1e-14)
    # identical keys: uniform weights -> mean of the values
    kk = np.broadcast_to(k[:, :, :1], k.shape).copy()
    np.testing.assert_allclose(O.attention(q, kk, v),
                               np.broadcast_to(v.mean(axis=2, keepdims=True), v.shape), rtol=1e-12)


def test_timestep_embedding_closed_form():
    e0 = O.timestep_embedding(0.0)
    np.testing.assert_array_equal(e0, np.concatenate([np.ones(128), np.zeros(128)]))
    s = 734.0
    e = O.timestep_embedding(s)
    assert e[0] == math.cos(s) and e[128] == math.sin(s)           # f_0 = 1
    np.testing.assert_allclose(e[64], math.cos(s / 100.0), rtol=1e-12)  # f_64 = 10^-2
    np.testing.assert_allclose(e[128 + 127], math.sin(s * 10000.0 ** (-127 / 128)), rtol=1e-12)


@pytest.mark.parametrize("lat,patch", [((4, 1, 8, 6), (1, 2, 2)), ((3, 4, 6, 4), (2, 2, 2)),
                                       ((2, 3, 4, 6), (1, 2, 3))])
def test_patchify_is_a_strided_convolution(lat, patch):
    rng = np.random.default_rng(4)
    C, F, H, W = lat
    x = rng.standard_normal((2, C, F, H, W))
    Cout = 5
    w = rng.standard_normal((Cout, C * patch[0] * patch[1] * patch[2]))
    got = O.patchify(x, patch) @ w.T                                  # [B, N, Cout]
    ref = Fn.conv3d(_t(x), _t(w.reshape(Cout, C, *patch)), stride=patch)  # [B, Cout, F', H', W']
    ref = ref.reshape(2, Cout, -1).transpose(1, 2).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_unpatchify_brute_force():
    rng = np.random.default_rng(5)
    lat, patch = (3, 4, 6, 4), (2, 3, 2)
    C, F, H, W = lat
    pt, ph, pw = patch
    Fp, Hp, Wp = F // pt, H // ph, W // pw
    y = rng.standard_normal((2, Fp * Hp * Wp, pt * ph * pw * C))
    got = O.unpatchify(y, patch, lat)
    ref = np.zeros((2, C, F, H, W))
    for b in range(2):
        for f in range(Fp):
            for hy in range(Hp):
                for wx in range(Wp):
                    tok = (f * Hp + hy) * Wp + wx
                    for a in range(pt):
                        for bb in range(ph):
                            for c in range(pw):
                                for ch in range(C):
                                    feat = ((a * ph + bb) * pw + c) * C + ch
                                    ref[b, ch, f * pt + a, hy * ph + bb, wx * pw + c] = y[b, tok, feat]
    np.testing.assert_array_equal(got, ref)


def test_rel_l1_brute_force():
    rng = np.random.default_rng(6)
    hf = rng.standard_normal((3, 4, 5))
    hd = hf + 0.1 * rng.standard_normal((3, 4, 5))
    got = O.rel_l1(hd, hf, 1e-8)
    for b in range(3):
        num = sum(abs(float(hd[b].flat[i]) - float(hf[b].flat[i])) for i in range(20))
        den = sum(abs(float(hf[b].flat[i])) for i in range(20))
        assert abs(got[b] - num / (den + 1e-8)) <= 1e-14
    assert np.all(O.rel_l1(hf, hf, 1e-8) == 0.0)


# ----------------------------------------------------------------------------- rotary embedding

def _rope_x(B=2, H=3, N=7, d=16, seed=3):
    return np.random.default_rng(seed).standard_normal((B, H, N, d))


def test_rope_position_zero_is_identity():
    x = _rope_x()
    assert np.array_equal(O.rope(x, np.zeros((7, 3)), (4, 6, 6), 10000.0), x)


def test_rope_keeps_pair_norms_and_is_a_rotation_by_pos():
    # one pair per axis chunk of 2 dims: the angle is pos * theta^0 = pos radians
    x = np.zeros((1, 1, 1, 6))
    x[..., 0], x[..., 2], x[..., 4] = 1.0, 2.0, 3.0
    pos = np.array([[1.0, 2.0, 3.0]])
    y = O.rope(x, pos, (2, 2, 2), 10000.0)
    np.testing.assert_allclose(y[0, 0, 0], [np.cos(1), np.sin(1), 2 * np.cos(2), 2 * np.sin(2),
                                            3 * np.cos(3), 3 * np.sin(3)], rtol=0, atol=1e-15)
    x = _rope_x(d=16)
    pos = np.random.default_rng(4).integers(0, 40, (7, 3)).astype(float)
    y = O.rope(x, pos, (4, 6, 6), 10000.0)
    np.testing.assert_allclose(np.hypot(y[..., 0::2], y[..., 1::2]), np.hypot(x[..., 0::2], x[..., 1::2]),
                               rtol=1e-12)


def test_rope_scores_depend_only_on_relative_positions():
    # q . k after rotation at positions p and p' equals the same at p + s and p' + s, for
    # any shift s per axis: the property rotary embeddings are built for
    rng = np.random.default_rng(5)
    q, k = rng.standard_normal((1, 1, 1, 16)), rng.standard_normal((1, 1, 1, 16))
    p, pp = np.array([[3.0, 5.0, 7.0]]), np.array([[1.0, 9.0, 2.0]])
    sft = np.array([[4.0, -2.0, 11.0]])
    dot = lambda a, b: float((a * b).sum())
    axes, th = (4, 6, 6), 10000.0
    d0 = dot(O.rope(q, p, axes, th), O.rope(k, pp, axes, th))
    d1 = dot(O.rope(q, p + sft, axes, th), O.rope(k, pp + sft, axes, th))
    assert abs(d0 - d1) < 1e-12 and abs(d0 - dot(q, k)) > 1e-3


def test_rope_positions_of_text_and_image_rows():
    cfg = dict(lat=(4, 2, 6, 8), patch=(1, 2, 2), n_txt=3)
    pos = O.rope_positions(cfg)
    assert pos.shape == (3 + 2 * 3 * 4, 3)
    assert np.all(pos[:3] == 0)
    np.testing.assert_array_equal(pos[3], [0, 0, 0])
    np.testing.assert_array_equal(pos[3 + 5], [0, 1, 1])          # token 5 of a 3 x 4 grid
    np.testing.assert_array_equal(pos[3 + 12 + 11], [1, 2, 3])    # last token of frame 1
