"""GPU parity of the exact block (Eq. 1) through ff_block_exact: element-wise against the
oracle at small ragged shapes (several tiles plus tails in every GEMM dimension, head dims
64 and 72, token tails), and on sampled rows at the workloads' full shapes."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline
from gpu_util import TOL, dev, host, need_gpu, say

pytestmark = pytest.mark.gpu


def ragged_cfg(kind, dtype, d=64, H=5, n_txt=0, B=2, lat=(4, 1, 20, 20), mlp_ratio=2):
    C = H * d
    kinds = [kind]
    n_img = (lat[1]) * (lat[2] // 2) * (lat[3] // 2)
    return dict(name="ragged", kinds=kinds, C=C, H=H, d=d, mlp=mlp_ratio * C, n_img=n_img, n_txt=n_txt, B=B,
                lat=lat, patch=(1, 2, 2), dtype=dtype, T=4, R=2, K=1, S=2, sites=[], site_rule="fixed",
                ln_eps=1e-6, rel_eps=1e-8)


def run_block(cfg, W, u_np, c_np, rows=None):
    dt = pipeline.torch_dtype(cfg)
    sets = [W["txt"], W["img"]] if cfg["kinds"][0] == synth.MMDIT_DOUBLE else [W]
    tens = [{k: dev(v, dt) for k, v in s.items()} for s in sets]
    lw = abi.ff_layer_weights()
    for si, s in enumerate(tens):
        for k, t in s.items():
            setattr(lw.s[si], k, t.data_ptr())
    m = pipeline.model_desc(cfg)
    ws_bytes = abi.ff_workspace_bytes(m)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    u = dev(u_np, dt)
    c = dev(c_np, torch.float32)
    h = torch.empty_like(u)
    abi.ff_block_exact(m, 0, lw, c.data_ptr(), u.data_ptr(), h.data_ptr(), ws.data_ptr(), ws_bytes)
    torch.cuda.synchronize()
    h2 = torch.empty_like(u)
    abi.ff_block_exact(m, 0, lw, c.data_ptr(), u.data_ptr(), h2.data_ptr(), ws.data_ptr(), ws_bytes)
    torch.cuda.synchronize()
    assert torch.equal(h, h2), "exact block is not deterministic"
    return host(h)


def boosted(W, kind):
    # larger modulation weights make every gate O(1) so that each branch is visible in h - u
    def b(s):
        s = dict(s)
        s["mod_w"] = (s["mod_w"] * 8).astype(np.float32)
        return s
    return {k: b(v) for k, v in W.items()} if kind == synth.MMDIT_DOUBLE else b(W)


def check_block(cfg, W, seed=0, rows=None, tol=None):
    kind = cfg["kinds"][0]
    bf = cfg["dtype"] == synth.BF16
    B, N, C = cfg["B"], cfg["n_img"] + cfg["n_txt"], cfg["C"]
    u = synth.normal((B, N, C), 300 + seed, bf16=bf)
    c = synth.normal((B, C), 400 + seed)
    got = run_block(cfg, W, u, c)
    u64 = u.astype(np.float64)
    cs = O.silu(c.astype(np.float64))
    ref = O.block(kind, u64, cs, W, cfg, rows=rows)
    if bf:
        ref = O.round_bf16(ref)
    g = got if rows is None else got[:, rows]
    uu = u64 if rows is None else u64[:, rows]
    err = O.max_rel_err(g - uu, ref - uu)       # error relative to the block's own update h - u
    tol = TOL[cfg["dtype"]] if tol is None else tol
    say(f"  block kind={kind} dtype={cfg['dtype']} B={B} N={N} C={C} d={cfg['d']}: err(h-u)={err:.3e} tol={tol}")
    assert err <= tol, err
    return err


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
@pytest.mark.parametrize("d,H", [(8, 40), (40, 8), (64, 5), (72, 5), (96, 5)])
def test_dit_block_ragged(dtype, d, H):
    # head dims from the smallest the boundary accepts (8, zero-padded to the 64-wide
    # attention tile) through the 80- and 96-wide tiles.  The small dims take many heads:
    # at C = 40 the block's update h - u is so small against h (0.12 against 3.9) that one
    # bf16 step of the stored output is 13 % of it, which the update-relative error
    # cannot tell from a wrong result.
    need_gpu()
    cfg = ragged_cfg(synth.DIT, dtype, d=d, H=H)
    W = boosted(synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.1), synth.DIT)
    say(f"dit ragged dtype={dtype} d={d}")
    check_block(cfg, W)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
@pytest.mark.parametrize("B", [9, 16, 27, 32])
def test_dit_block_batch_groups(dtype, B):
    # the modulation GEMV takes samples in groups of 8 (one weight read for all groups on
    # MFMA, one launch per group in fp32): full, ragged and the largest batch
    need_gpu()
    cfg = ragged_cfg(synth.DIT, dtype, d=64, H=3, B=B, lat=(4, 1, 8, 10))
    W = boosted(synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.1), synth.DIT)
    say(f"dit batch groups dtype={dtype} B={B}")
    check_block(cfg, W)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
@pytest.mark.parametrize("kind", [synth.MMDIT_DOUBLE, synth.MMDIT_SINGLE])
def test_mmdit_blocks_ragged(dtype, kind):
    need_gpu()
    cfg = ragged_cfg(kind, dtype, d=64, H=3, n_txt=13, lat=(4, 1, 18, 22))
    W = boosted(synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.2), kind)
    say(f"mmdit ragged kind={kind} dtype={dtype}")
    check_block(cfg, W, seed=kind)


def test_tiny_shape_block_fp32():
    need_gpu()
    cfg = synth.get_config("tiny", kinds=[synth.DIT])
    W = synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.1)
    say("tiny block")
    check_block(cfg, W)


def test_dit_xl2_block_full_shape():
    need_gpu()
    cfg = synth.get_config("dit_xl2", kinds=[synth.DIT])
    W = synth.make_layer_weights(cfg, 0, bias_std=0.02)
    say("dit_xl2 full block B=8 N=256 C=1152 d=72")
    check_block(cfg, W)


SAMPLE_ROWS = {
    "flux": [0, 1, 511, 512, 513, 2000, 4095, 4607],
    "qwen": [0, 255, 256, 257, 3000, 4351],
    "hunyuan": [0, 255, 256, 300, 7000, 14309, 14565],
}


@pytest.mark.parametrize("name,kind", [("flux", synth.MMDIT_SINGLE), ("flux", synth.MMDIT_DOUBLE),
                                       ("qwen", synth.MMDIT_DOUBLE), ("hunyuan", synth.MMDIT_DOUBLE)])
def test_mmdit_block_full_shape_sampled_rows(name, kind):
    need_gpu()
    cfg = synth.get_config(name, kinds=[kind])
    W = synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.1)
    say(f"{name} full block kind={kind} N={cfg['n_img'] + cfg['n_txt']} (sampled rows)")
    check_block(cfg, W, rows=np.array(SAMPLE_ROWS[name]))


def test_dit_block_gemm_tile_paths():
    """A DiT block whose GEMMs take the 32-wide K-stage paths: qkv and fc1 256x256 tiles
    (K = 2080 is not a multiple of 64), proj 128x128; fc2 (K = 8320, 64-wide stages) 128x96
    tiles with two k groups of waves; attention with head dim 104."""
    need_gpu()
    cfg = ragged_cfg(synth.DIT, synth.BF16, d=104, H=20, B=2, lat=(4, 1, 64, 64), mlp_ratio=4)
    W = boosted(synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.1), synth.DIT)
    say("dit block C=2080 d=104 N=1024 B=2 (sampled rows)")
    check_block(cfg, W, rows=np.array([0, 1, 255, 256, 511, 700, 1022, 1023]))


def test_dit_block_ragged_wide_tiles():
    """A DiT block with 2000 token rows (ragged against both the 256- and 128-row tiles):
    fc1 (N = 4608) takes 256x192 tiles, proj and fc2 128x96 tiles with four 64-wide K
    stages and two k groups of waves, qkv two 128x128 tiles per CU."""
    need_gpu()
    cfg = ragged_cfg(synth.DIT, synth.BF16, d=72, H=16, B=4, lat=(4, 1, 50, 40), mlp_ratio=4)
    W = boosted(synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.1), synth.DIT)
    say("dit block C=1152 d=72 N=500 B=4 (sampled rows)")
    check_block(cfg, W, rows=np.array([0, 1, 127, 128, 255, 256, 420, 450, 498, 499]))


def test_dit_block_c2048_tiles():
    """A DiT block with C = 2048 (16 heads of 128) and 2048 rows: qkv takes 256x192 and fc1
    256x256 tiles with 64-wide stages, proj and fc2 (N = 2048, 256 tiles) one 128x128 tile
    per CU with four 64-wide stages and two k groups; attention with head dim 128."""
    need_gpu()
    cfg = ragged_cfg(synth.DIT, synth.BF16, d=128, H=16, B=2, lat=(4, 1, 64, 64), mlp_ratio=4)
    W = boosted(synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.1), synth.DIT)
    say("dit block C=2048 d=128 N=1024 B=2 (sampled rows)")
    check_block(cfg, W, rows=np.array([0, 1, 127, 128, 511, 777, 1023]))



def test_dit_block_attention_wide_ragged():
    """Head dim 128 on the 8-wavefront attention grid (4 query blocks x 16 heads x 4
    samples = 256 workgroups, 128-key tiles): 1000 tokens per sample, so the last query
    block holds 232 queries and the last key tile 104 keys."""
    need_gpu()
    cfg = ragged_cfg(synth.DIT, synth.BF16, d=128, H=16, B=4, lat=(4, 1, 50, 80), mlp_ratio=4)
    W = boosted(synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.1), synth.DIT)
    say("dit block C=2048 d=128 N=1000 B=4 (sampled rows)")
    check_block(cfg, W, rows=np.array([0, 1, 255, 256, 511, 767, 768, 959, 960, 998, 999]))


def test_dit_block_narrow_tiles():
    """A DiT block with 510 token rows (two samples of 255 tokens; the last 128-row tile
    holds 126): qkv, proj and fc2 take 128x64 tiles and fc1 128x96 tiles, both with two k
    groups of waves, so the gated epilogue runs on the 128x64 path too."""
    need_gpu()
    cfg = ragged_cfg(synth.DIT, synth.BF16, d=72, H=16, B=2, lat=(4, 1, 30, 34), mlp_ratio=4)
    W = boosted(synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.1), synth.DIT)
    say("dit block C=1152 d=72 N=255 B=2")
    check_block(cfg, W)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
@pytest.mark.parametrize("kind", [synth.MMDIT_DOUBLE, synth.MMDIT_SINGLE])
def test_mmdit_blocks_rope(dtype, kind):
    """Rotary embedding of q and k (3-axis ids: text rows 0, image rows (frame, row,
    column)) on a two-frame latent with ragged text and image rows."""
    need_gpu()
    cfg = ragged_cfg(kind, dtype, d=64, H=3, n_txt=13, lat=(4, 2, 18, 22))
    cfg["rope_axes"], cfg["rope_theta"] = (16, 24, 24), 10000.0
    W = boosted(synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.2), kind)
    say(f"mmdit rope kind={kind} dtype={dtype}")
    check_block(cfg, W, seed=kind)


@pytest.mark.parametrize("kind", [synth.MMDIT_SINGLE, synth.MMDIT_DOUBLE])
def test_flux_block_rope_full_shape_sampled_rows(kind):
    need_gpu()
    cfg = synth.get_config("flux", kinds=[kind])
    cfg["rope_axes"], cfg["rope_theta"] = (16, 56, 56), 10000.0
    W = synth.make_layer_weights(cfg, 0, bias_std=0.02, gain_std=0.1)
    say(f"flux rope full block kind={kind} (sampled rows)")
    check_block(cfg, W, rows=np.array(SAMPLE_ROWS["flux"]))
