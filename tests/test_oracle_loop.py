"""Pins for the oracle's schedule and whole loop: counter closed forms per workload,
the invariants the paper states (Sec. 3.3 and Eq. 5) and sampler closed forms."""
import numpy as np
import pytest

import oracle as O
import synth


@pytest.mark.parametrize("name,refresh,paid", [("tiny", 4, 12), ("dit_xl2", 10, 80),
                                               ("flux", 9, 123), ("qwen", 10, 160),
                                               ("hunyuan", 10, 80)])
def test_counter_closed_forms(name, refresh, paid):
    cfg = synth.get_config(name)
    T, R, L = cfg["T"], cfg["R"], len(cfg["kinds"])
    mask = synth.site_mask(cfg)
    assert refresh == -(-T // R)
    cached = [i for i in range(T) if i % R]
    for mode in (O.VERIFY, O.FEATFIX, O.EXACT_ONLY, O.DRAFT, O.VANILLA, O.TOKENS_PARTIAL, O.CHANNELS_PARTIAL,
                 O.RECOMPUTE):
        p = O.make_plan(T, L, R, cfg["K"], cfg["S"], mask, mode)
        c = p["counts"]
        if mode == O.VANILLA:
            assert c == {"n_full_refresh": T, "n_paid_checks": 0, "n_forwarded": 0, "n_recomputed": 0}
            continue
        assert c["n_full_refresh"] == refresh
        if mode == O.RECOMPUTE:
            # the first site of each checked step is paid, the layers after it recomputed
            firsts = [int(np.argmax(mask[i])) for i in cached if mask[i].any()]
            assert c["n_paid_checks"] == c["n_forwarded"] == len(firsts)
            assert c["n_recomputed"] == sum(L - 1 - f for f in firsts)
            continue
        expect_paid = 0 if mode == O.DRAFT else paid
        assert c["n_paid_checks"] == expect_paid
        assert c["n_forwarded"] == (expect_paid if mode in O.FORWARDING_MODES else 0)
        assert c["n_recomputed"] == 0
        assert expect_paid == (0 if mode == O.DRAFT else int(sum(mask[i].sum() for i in cached)))


def test_splitmix64_reference_values_and_qwen_sites():
    g = synth.splitmix64_stream(0)
    assert [next(g) for _ in range(3)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    s = synth.sites_of(synth.get_config("qwen"))
    assert len(s) == 4 and len(set(s)) == 4 and all(0 <= x < 60 for x in s) and s == sorted(s)


def test_plan_slots_follow_the_ring():
    T, L, R, K, S = 23, 3, 4, 2, 3
    mask = np.zeros((T, L), np.uint8)
    mask[:, 1] = 1
    p = O.make_plan(T, L, R, K, S, mask, O.FEATFIX)
    for i in range(T):
        j = i // R
        assert p["refresh_ord"][i] == j
        if i % R == 0:
            assert p["write_slot"][i] == j % S and (p["read_slots"][i] == -1).all()
            assert (p["action"][i] == O.EXACT).all()
        else:
            ke = min(K, j)
            assert p["k_eff"][i] == ke and p["write_slot"][i] == -1
            assert list(p["read_slots"][i][:ke + 1]) == [(j - m) % S for m in range(ke + 1)]
            assert (p["read_slots"][i][ke + 1:] == -1).all()
            assert list(p["action"][i]) == [O.DRAFT_ACT, O.SITE, O.DRAFT_ACT]


def tiny_setup(**over):
    cfg = synth.get_config("tiny", **over)
    W = synth.make_weights(cfg, bias_std=0.02, gain_std=0.1)
    inp = synth.make_inputs(cfg)
    return cfg, W, inp


def test_featfix_equals_exact_only_at_every_layer():
    cfg, W, inp = tiny_setup()
    mask = synth.site_mask(cfg)
    ta, tb = [], []
    a = O.run(cfg, O.FEATFIX, inp, W, mask, trace=ta)
    b = O.run(cfg, O.EXACT_ONLY, inp, W, mask, trace=tb)
    np.testing.assert_array_equal(a["x"], b["x"])
    for x, y in zip(ta, tb):
        np.testing.assert_array_equal(x, y)
    assert a["counts"] == b["counts"] and b["audit"] == {}
    assert len(a["audit"]) == a["counts"]["n_paid_checks"]


def test_verify_equals_draft_and_logs_the_same_checks():
    cfg, W, inp = tiny_setup()
    mask = synth.site_mask(cfg)
    v = O.run(cfg, O.VERIFY, inp, W, mask)
    d = O.run(cfg, O.DRAFT, inp, W, mask)
    f = O.run(cfg, O.FEATFIX, inp, W, mask)
    np.testing.assert_array_equal(v["x"], d["x"])
    assert v["counts"]["n_paid_checks"] == f["counts"]["n_paid_checks"] == 12
    assert v["counts"]["n_forwarded"] == 0 and f["counts"]["n_forwarded"] == 12
    # the first paid check sees the same incoming state in both arms
    first = min(f["audit"])
    np.testing.assert_array_equal(v["audit"][first], f["audit"][first])
    assert not np.array_equal(v["x"], f["x"])


def test_all_sites_and_r1_reproduce_vanilla():
    cfg, W, inp = tiny_setup()
    van = O.run(cfg, O.VANILLA, inp, W, synth.site_mask(cfg))
    ones = np.ones((cfg["T"], 4), np.uint8)
    np.testing.assert_array_equal(O.run(cfg, O.FEATFIX, inp, W, ones)["x"], van["x"])
    np.testing.assert_array_equal(O.run(cfg, O.EXACT_ONLY, inp, W, ones)["x"], van["x"])
    cfg1 = dict(cfg, R=1)
    np.testing.assert_array_equal(O.run(cfg1, O.FEATFIX, inp, W, synth.site_mask(cfg1))["x"], van["x"])


def test_site_output_is_the_exact_block_of_the_same_input():
    # Eq. 5: at a site the forwarded tensor is B_l(u) for the incoming u -> residual exactly 0
    cfg, W, inp = tiny_setup()
    mask = synth.site_mask(cfg)
    tr = []
    O.run(cfg, O.FEATFIX, inp, W, mask, trace=tr)
    L = 4
    i, l = 1, 1        # first cached step, first site
    u = tr[i * L + l - 1]
    cs = O.silu(O.conditioning(inp["c"], 1.0 - i / cfg["T"], W[1]))
    np.testing.assert_array_equal(tr[i * L + l], O.block(O.DIT, u, cs, W[0][l], cfg))


def test_euler_closed_form_with_constant_velocity():
    cfg, W, inp = tiny_setup()
    layers, G = W
    G = dict(G)
    G["f_w"] = np.zeros_like(G["f_w"])
    G["f_b"] = np.random.default_rng(0).standard_normal(G["f_b"].shape).astype(np.float32)
    out = O.run(cfg, O.FEATFIX, inp, (layers, G), synth.site_mask(cfg))
    v = O.unpatchify(np.broadcast_to(G["f_b"].astype(np.float64), (1, 64, 16)), cfg["patch"], cfg["lat"])
    np.testing.assert_allclose(out["x"], inp["x"] - v, rtol=1e-13, atol=1e-13)   # sum of dt = -1


def test_output_mode_order_zero_reuses_block_outputs():
    # feature_mode OUTPUT with K=0: the draft of layer l is h_l at the last refresh (reuse)
    cfg, W, inp = tiny_setup(K=0, S=1)
    mask = np.zeros((cfg["T"], 4), np.uint8)
    tr = []
    O.run(cfg, O.DRAFT, inp, W, mask, feature_mode=O.OUTPUT, trace=tr)
    L, R = 4, cfg["R"]
    for i in range(cfg["T"]):
        if i % R:
            s = (i // R) * R
            for l in range(L):
                np.testing.assert_array_equal(tr[i * L + l], tr[s * L + l])


def test_bf16_stream_is_bf16_valued():
    cfg = synth.get_config("tiny", dtype=synth.BF16, T=4)
    W = synth.make_weights(cfg)
    inp = synth.make_inputs(cfg)
    tr = []
    O.run(cfg, O.FEATFIX, inp, W, synth.site_mask(cfg), trace=tr)
    for x in tr:
        np.testing.assert_array_equal(O.round_bf16(x), x)
