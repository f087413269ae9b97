"""Seeded synthetic inputs for the cached-DiT denoising workloads.

This module is shared by the CPU oracle's tests and by the GPU path's tests and
benchmark.  It holds workload descriptions (shapes, schedule parameters, site
sets) and random-number draws only: none of the method's arithmetic lives here.

Seeds (named sub-seeds of numpy's PCG64): weights 0, latent 1, conditioning 2,
text tokens 3.  The Qwen-like site set is drawn with SplitMix64 (Steele, Lea and
Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014) seeded 0.

The paper's own workloads (FLUX.1-dev on DrawBench prompts, Qwen-Image,
HunyuanVideo-1.5, DiT-XL/2 on ImageNet-256) need trained weights, encoders and
datasets that are not available; these synthetic inputs keep their shapes:
text prompts become N(0,1) text tokens, class labels an N(0,1) conditioning
vector, and the initial noise latent is N(0,1) as in the real sampler.
"""
from __future__ import annotations

import copy
import numpy as np

DIT, MMDIT_DOUBLE, MMDIT_SINGLE = 0, 1, 2
F32, BF16 = 0, 1
VANILLA, DRAFT, VERIFY, FEATFIX, EXACT_ONLY = 0, 1, 2, 3, 4
TOKENS_PARTIAL, CHANNELS_PARTIAL, RECOMPUTE = 5, 6, 7
MODE_NAMES = {"vanilla": VANILLA, "draft": DRAFT, "verify": VERIFY,
              "featfix": FEATFIX, "exact_only": EXACT_ONLY, "tokens_partial": TOKENS_PARTIAL,
              "channels_partial": CHANNELS_PARTIAL, "recompute": RECOMPUTE}
RESIDUAL, OUTPUT = 0, 1

WEIGHT_STD = 0.02
TEMB_DIM = 256


def _cfg(name, kinds, C, H, d, mlp, n_img, n_txt, B, lat, patch, dtype, T, R, K, S, sites,
         site_rule="fixed"):
    return dict(name=name, kinds=list(kinds), C=C, H=H, d=d, mlp=mlp, n_img=n_img,
                n_txt=n_txt, B=B, lat=tuple(lat), patch=tuple(patch), dtype=dtype, T=T, R=R,
                K=K, S=S, sites=list(sites), site_rule=site_rule, ln_eps=1e-6, rel_eps=1e-8)


# Workloads (hidden C, heads H x head dim d, MLP hidden, tokens, batch,
# latent [C_lat, F, H, W] and patch (pt, ph, pw), schedule T/R/K/S, 0-based sites).
CONFIGS = {
    # 4-block DiT, fp32: the small case used for element-wise parity of the whole loop.
    "tiny": _cfg("tiny", [DIT] * 4, 256, 4, 64, 1024, 64, 0, 1, (4, 1, 16, 16), (1, 2, 2),
                 F32, 10, 3, 1, 2, [1, 3]),
    # DiT-XL/2 shape: 28 blocks, 1152 wide, 16x72 heads, 256 tokens, batch 8.
    "dit_xl2": _cfg("dit_xl2", [DIT] * 28, 1152, 16, 72, 4608, 256, 0, 8, (4, 1, 32, 32),
                    (1, 2, 2), BF16, 50, 5, 2, 3, [13, 27]),
    # FLUX-like MMDiT: 19 double + 38 single blocks, 4096 image + 512 text tokens.
    "flux": _cfg("flux", [MMDIT_DOUBLE] * 19 + [MMDIT_SINGLE] * 38, 3072, 24, 128, 12288,
                 4096, 512, 1, (16, 1, 128, 128), (1, 2, 2), BF16, 50, 6, 1, 2, [18, 37, 56]),
    # Qwen-Image-like: 60 double-stream blocks, 4 sites drawn from SplitMix64(0).
    "qwen": _cfg("qwen", [MMDIT_DOUBLE] * 60, 3072, 24, 128, 12288, 4096, 256, 1,
                 (16, 1, 128, 128), (1, 2, 2), BF16, 50, 5, 2, 3, [], site_rule="splitmix4"),
    # HunyuanVideo-like: 54 double-stream blocks over 9x30x53 video + 256 text tokens.
    "hunyuan": _cfg("hunyuan", [MMDIT_DOUBLE] * 54, 2048, 16, 128, 8192, 14310, 256, 1,
                    (16, 9, 60, 106), (1, 2, 2), BF16, 50, 5, 1, 3, [26, 53]),
}


def get_config(name: str, **overrides) -> dict:
    cfg = copy.deepcopy(CONFIGS[name])
    cfg.update(overrides)
    return cfg


def derived(cfg: dict) -> dict:
    """Shape quantities that follow from a workload description."""
    c_lat, F, Hh, W = cfg["lat"]
    pt, ph, pw = cfg["patch"]
    n_img = (F // pt) * (Hh // ph) * (W // pw)
    assert n_img == cfg["n_img"], (n_img, cfg["n_img"])
    return dict(L=len(cfg["kinds"]), N=cfg["n_img"] + cfg["n_txt"], P=pt * ph * pw * c_lat,
                grid=(F // pt, Hh // ph, W // pw))


# ----------------------------------------------------------------------------- rng helpers

def splitmix64_stream(seed: int):
    """SplitMix64 generator (published constants), yields 64-bit ints."""
    mask = (1 << 64) - 1
    state = seed & mask
    while True:
        state = (state + 0x9E3779B97F4A7C15) & mask
        z = state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & mask
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & mask
        yield z ^ (z >> 31)


def splitmix_sites(n_layers: int, n_pick: int, seed: int = 0) -> list:
    """Partial Fisher-Yates over 0..n_layers-1 driven by SplitMix64; first n_pick, sorted."""
    g = splitmix64_stream(seed)
    perm = list(range(n_layers))
    for i in range(n_pick):
        j = i + (next(g) % (n_layers - i))
        perm[i], perm[j] = perm[j], perm[i]
    return sorted(perm[:n_pick])


def sites_of(cfg: dict) -> list:
    if cfg["site_rule"] == "splitmix4":
        return splitmix_sites(len(cfg["kinds"]), 4, 0)
    return list(cfg["sites"])


def site_mask(cfg: dict, sites=None) -> np.ndarray:
    """uint8 [T, L], step-major: the fixed site set on every step (refresh bits are ignored
    by the schedule)."""
    T, L = cfg["T"], len(cfg["kinds"])
    m = np.zeros((T, L), np.uint8)
    for l in (sites_of(cfg) if sites is None else sites):
        m[:, l] = 1
    return m


def to_bf16_values(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns fp32 holding bf16 values."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    r = (u >> 16) & np.uint32(1)          # finite values cannot overflow uint32 below
    r += np.uint32(0x7FFF)
    r += u
    r &= np.uint32(0xFFFF0000)
    out = r.view(np.float32)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = np.nan
    return out


def _rng(*key):
    return np.random.default_rng(list(key))


def _normal(shape, std, *key):
    a = _rng(*key).standard_normal(shape, dtype=np.float32)
    a *= np.float32(std)
    return a


# Tensor ids inside one layer's weight set; used to seed one PCG64 stream per tensor so a
# single layer can be generated without generating the others.
_DIT_FIELDS = ("mod", "qkv", "o", "fc1", "fc2")
_SINGLE_FIELDS = ("mod", "lin1", "lin2")


def layer_shapes(cfg: dict, kind: int) -> dict:
    C, M, d = cfg["C"], cfg["mlp"], cfg["d"]
    if kind == DIT or kind == MMDIT_DOUBLE:
        return {"mod": (6 * C, C), "qkv": (3 * C, C), "o": (C, C), "fc1": (M, C), "fc2": (C, M)}
    return {"mod": (3 * C, C), "lin1": (3 * C + M, C), "lin2": (C, C + M)}


def make_layer_weights(cfg: dict, layer: int, seed: int = 0, bias_std: float = 0.0,
                       gain_std: float = 0.0) -> dict:
    """One layer's weights.  Matrices are [out, in] with N(0, 0.02^2) entries; biases are
    zero and norm gains one unless bias_std / gain_std ask for perturbed values (used by
    parity tests so that a dropped bias or gain cannot go unnoticed)."""
    kind = cfg["kinds"][layer]
    bf16 = cfg["dtype"] == BF16
    fix = to_bf16_values if bf16 else (lambda a: a)
    d = cfg["d"]

    def one_set(stream: int):
        out = {}
        for t, (name, shp) in enumerate(layer_shapes(cfg, kind).items()):
            out[name + "_w"] = fix(_normal(shp, WEIGHT_STD, seed, 1000 + layer, stream, t, 0))
            if bias_std > 0:
                out[name + "_b"] = fix(_normal((shp[0],), bias_std, seed, 1000 + layer, stream, t, 1))
            else:
                out[name + "_b"] = np.zeros((shp[0],), np.float32)
        if kind != DIT:
            for t, g in enumerate(("q_g", "k_g")):
                if gain_std > 0:
                    out[g] = fix(1.0 + _normal((d,), gain_std, seed, 1000 + layer, stream, 50 + t, 2))
                else:
                    out[g] = np.ones((d,), np.float32)
        return out

    if kind == MMDIT_DOUBLE:
        return {"txt": one_set(0), "img": one_set(1)}
    return one_set(0)


def make_global_weights(cfg: dict, seed: int = 0, bias_std: float = 0.0) -> dict:
    """Time-embedding MLP, patch embedding and final (adaLN + linear) layer."""
    C = cfg["C"]
    P = derived(cfg)["P"]
    bf16 = cfg["dtype"] == BF16
    fix = to_bf16_values if bf16 else (lambda a: a)
    shapes = {"t1": (C, TEMB_DIM), "t2": (C, C), "pe": (C, P), "fmod": (2 * C, C), "f": (P, C)}
    out = {}
    for t, (name, shp) in enumerate(shapes.items()):
        out[name + "_w"] = fix(_normal(shp, WEIGHT_STD, seed, 7, t, 0))
        if bias_std > 0:
            out[name + "_b"] = fix(_normal((shp[0],), bias_std, seed, 7, t, 1))
        else:
            out[name + "_b"] = np.zeros((shp[0],), np.float32)
    return out


def make_weights(cfg: dict, seed: int = 0, bias_std: float = 0.0, gain_std: float = 0.0):
    return ([make_layer_weights(cfg, l, seed, bias_std, gain_std) for l in range(len(cfg["kinds"]))],
            make_global_weights(cfg, seed, bias_std))


def make_inputs(cfg: dict, seeds=(1, 2, 3)) -> dict:
    """Initial latent x (fp32, N(0,1)), conditioning vector c [B, C] and text tokens
    [B, N_txt, C] (both N(0,1), rounded to bf16 values in bf16 workloads).  With
    cfg["cfg_pairs"] the B model rows are B/2 guided pairs, so x holds B/2 latents."""
    B, C = cfg["B"], cfg["C"]
    c_lat, F, Hh, W = cfg["lat"]
    bf16 = cfg["dtype"] == BF16
    fix = to_bf16_values if bf16 else (lambda a: a)
    Bx = B // 2 if cfg.get("cfg_pairs") else B
    x = _rng(seeds[0]).standard_normal((Bx, c_lat, F, Hh, W), dtype=np.float32)
    c = fix(_rng(seeds[1]).standard_normal((B, C), dtype=np.float32))
    txt = fix(_rng(seeds[2]).standard_normal((B, cfg["n_txt"], C), dtype=np.float32))
    return {"x": x, "c": c, "txt": txt}


def normal(shape, seed, std=1.0, bf16=False):
    """Generic seeded N(0, std^2) fp32 tensor (optionally bf16-valued) for kernel tests."""
    a = _normal(shape, std, 99, seed)
    return to_bf16_values(a) if bf16 else a


def reduced_stack(name: str) -> dict:
    """Reduced-depth, full-width parity stacks of the MMDiT workloads: every block at the
    workload's full hidden size, heads, MLP width, token counts and batch, fewer blocks
    and steps (refresh every 3 steps), sites by the workload's own rule applied to the
    shorter stack, and enough blocks that a cached step has a run of two or more drafted
    layers (the runs the history sums stand in for).
      flux:    3 double + 5 single; sites last double, middle single, last single {2, 4, 7}
      qwen:    4 double, K = 2, S = 3, 1 site drawn by SplitMix64(0) as the 60-layer rule
               draws 4; T = 8 puts step 7 at k_eff = 2
      hunyuan: 5 double over 14 310 + 256 tokens, sites middle (L/2 - 1) and last {1, 4};
               T = 5 (refreshes 0 and 3)"""
    if name == "flux":
        return get_config("flux", kinds=[MMDIT_DOUBLE] * 3 + [MMDIT_SINGLE] * 5, T=8, R=3, sites=[2, 4, 7])
    if name == "qwen":
        return get_config("qwen", kinds=[MMDIT_DOUBLE] * 4, T=8, R=3, site_rule="fixed",
                          sites=splitmix_sites(4, 1, 0))
    if name == "hunyuan":
        return get_config("hunyuan", kinds=[MMDIT_DOUBLE] * 5, T=5, R=3, sites=[1, 4])
    raise KeyError(name)
