"""Device-side plumbing around the C ABI: weights, cache and workspace live in torch
device tensors (PyTorch is used for memory and streams only) and every step runs through
``ff_denoise_step``.

    dm = DeviceModel.from_host(cfg, layer_weights, global_weights)     # or DeviceModel.random(cfg)
    run = Runner(dm, mode=abi.FF_FEATFIX, mask=site_mask)
    x_T, audit, counts = run.run(x0, cond, txt)
"""
from __future__ import annotations

import ctypes as C

import numpy as np
import torch

from . import abi

_DEV = "cuda"


def torch_dtype(cfg):
    return torch.bfloat16 if cfg["dtype"] == abi.FF_BF16 else torch.float32


def model_desc(cfg):
    """ff_model_desc for a workload description (keeps its kinds array alive on the struct)."""
    kinds = (C.c_int32 * len(cfg["kinds"]))(*cfg["kinds"])
    c_lat, F, H, W = cfg["lat"]
    pt, ph, pw = cfg["patch"]
    m = abi.ff_model_desc(len(cfg["kinds"]), kinds, cfg["C"], cfg["H"], cfg["d"], cfg["mlp"], cfg["n_img"],
                          cfg["n_txt"], cfg["B"], c_lat, F, H, W, pt, ph, pw, cfg["dtype"], cfg["ln_eps"],
                          (C.c_int32 * 3)(*cfg.get("rope_axes", (0, 0, 0))), cfg.get("rope_theta", 10000.0),
                          cfg.get("cfg_pairs", 0), cfg.get("cfg_scale", 1.0))
    m._kinds = kinds
    return m


def _stream_shapes(cfg, kind):
    Cc, M, d = cfg["C"], cfg["mlp"], cfg["d"]
    if kind == abi.FF_MMDIT_SINGLE:
        shp = {"mod": (3 * Cc, Cc), "lin1": (3 * Cc + M, Cc), "lin2": (Cc, Cc + M)}
    else:
        shp = {"mod": (6 * Cc, Cc), "qkv": (3 * Cc, Cc), "o": (Cc, Cc), "fc1": (M, Cc), "fc2": (Cc, M)}
    out = {}
    for k, s in shp.items():
        out[k + "_w"] = s
        out[k + "_b"] = (s[0],)
    if kind != abi.FF_DIT:
        out["q_g"] = (d,)
        out["k_g"] = (d,)
    return out


def _global_shapes(cfg):
    Cc = cfg["C"]
    c_lat = cfg["lat"][0]
    P = cfg["patch"][0] * cfg["patch"][1] * cfg["patch"][2] * c_lat
    shp = {"t1": (Cc, abi.FF_TEMB_DIM), "t2": (Cc, Cc), "pe": (Cc, P), "fmod": (2 * Cc, Cc), "f": (P, Cc)}
    out = {}
    for k, s in shp.items():
        out[k + "_w"] = s
        out[k + "_b"] = (s[0],)
    return out


class DeviceModel:
    """Model weights resident in HBM, with the ABI structs that point at them."""

    def __init__(self, cfg, layer_tensors, global_tensors):
        self.cfg = cfg
        self.desc = model_desc(cfg)
        L = len(cfg["kinds"])
        self.layer_tensors = layer_tensors
        self.global_tensors = global_tensors
        self.lw = (abi.ff_layer_weights * L)()
        for l in range(L):
            sets = layer_tensors[l]
            for si, ws in enumerate(sets):
                for name, t in ws.items():
                    setattr(self.lw[l].s[si], name, t.data_ptr())
        self.g = abi.ff_global_weights(**{k: t.data_ptr() for k, t in global_tensors.items()})

    @staticmethod
    def _sets(cfg, l, W):
        return [W["txt"], W["img"]] if cfg["kinds"][l] == abi.FF_MMDIT_DOUBLE else [W]

    @classmethod
    def from_host(cls, cfg, layer_weights, global_weights, device=_DEV):
        """Upload host (numpy) weights; values are used exactly (bf16 workloads pass bf16 values)."""
        dt = torch_dtype(cfg)
        up = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device=device, dtype=dt)
        layers = [[{k: up(v) for k, v in s.items()} for s in cls._sets(cfg, l, W)]
                  for l, W in enumerate(layer_weights)]
        glob = {k: up(v) for k, v in global_weights.items()}
        return cls(cfg, layers, glob)

    @classmethod
    def random(cls, cfg, seed=0, device=_DEV, std=0.02):
        """Random-init weights generated on the device (for full-depth throughput runs):
        matrices N(0, std^2), biases zero, norm gains one."""
        dt = torch_dtype(cfg)
        g = torch.Generator(device=device)
        g.manual_seed(seed)

        def make(name, shp):
            if name.endswith("_b"):
                return torch.zeros(shp, dtype=dt, device=device)
            if name.endswith("_g"):
                return torch.ones(shp, dtype=dt, device=device)
            return (torch.randn(shp, generator=g, device=device, dtype=torch.float32) * std).to(dt)

        layers = []
        for l, kind in enumerate(cfg["kinds"]):
            n_sets = 2 if kind == abi.FF_MMDIT_DOUBLE else 1
            layers.append([{k: make(k, s) for k, s in _stream_shapes(cfg, kind).items()} for _ in range(n_sets)])
        glob = {k: make(k, s) for k, s in _global_shapes(cfg).items()}
        return cls(cfg, layers, glob)


class Runner:
    """A plan + cache + workspace + context for one mode of one model."""

    def __init__(self, dm: DeviceModel, mode, mask, feature_mode=abi.FF_RESIDUAL, T=None, R=None, K=None,
                 S=None, eps=None, tau=0.0, part_stride=2, hist_sums=False, cond_cache=False, device=_DEV):
        cfg = dm.cfg
        self.dm = dm
        self.T = cfg["T"] if T is None else T
        self.R = cfg["R"] if R is None else R
        self.K = cfg["K"] if K is None else K
        self.S = cfg["S"] if S is None else S
        self.L = len(cfg["kinds"])
        self.mode = mode
        self.sched = abi.ff_sched_desc(self.T, self.R, self.K, self.S, cfg["rel_eps"] if eps is None else eps,
                                       mode, feature_mode, tau, part_stride)
        self.plan = abi.ff_plan_build(self.sched, self.L, np.asarray(mask, np.uint8).reshape(-1))
        # Vanilla never reads or writes the history: it gets no cache
        self.cache_bytes = 0 if mode == abi.FF_VANILLA else abi.ff_cache_bytes(dm.desc, self.S)
        self.ws_bytes = abi.ff_workspace_bytes(dm.desc)
        self.cache = torch.empty(max(self.cache_bytes, 256), dtype=torch.uint8, device=device)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.ctx = abi.ff_ctx_create(dm.desc, dm.lw, dm.g, self.plan, self.cache.data_ptr(), self.cache_bytes,
                                     self.ws.data_ptr(), self.ws_bytes)
        # runs of drafted layers applied from per-run history sums formed at the refreshes
        self.hsum = None
        if hist_sums:
            nb = abi.ff_hist_sum_bytes(dm.desc, self.plan)
            if nb:
                self.hsum = torch.empty(nb, dtype=torch.uint8, device=device)
                abi.ff_ctx_hist_sums(self.ctx, self.hsum.data_ptr(), nb)
        # the conditioning of the whole schedule formed at step 0 (every step then passes
        # the same cond tensor)
        self.ccache = None
        if cond_cache:
            nb = abi.ff_cond_cache_bytes(dm.desc, self.plan)
            self.ccache = torch.empty(nb, dtype=torch.uint8, device=device)
            abi.ff_ctx_cond_cache(self.ctx, self.ccache.data_ptr(), nb)

    def export_plan(self):
        return abi.ff_plan_export(self.plan, self.T, self.L, self.K)

    def start(self, x0, audit=True):
        abi.ff_ctx_reset(self.ctx)
        cfg = self.dm.cfg
        x = x0.clone()
        a = torch.full((self.T * self.L * cfg["B"],), float("nan"), dtype=torch.float32, device=x0.device) \
            if audit else None
        return x, a

    def step(self, i, x, cond, txt=None, audit=None, stream=None):
        s = torch.cuda.current_stream().cuda_stream if stream is None else stream
        abi.ff_denoise_step(self.ctx, i, x.data_ptr(), cond.data_ptr(),
                            None if txt is None else txt.data_ptr(),
                            None if audit is None else audit.data_ptr(), s)

    def trace_into(self, buf):
        """Copy the stream after every layer of each step into buf ([L, B*N*C] model dtype
        tensor, or None to stop)."""
        abi.ff_ctx_trace(self.ctx, None if buf is None else buf.data_ptr(), 0 if buf is None else buf.numel() * buf.element_size())

    def step_kinds(self):
        """Realised kind of each step of the current run (-1 for steps not run yet)."""
        return abi.ff_ctx_step_kinds(self.ctx, self.T)

    def run(self, x0, cond, txt=None, audit=True):
        """Whole T-step loop; returns (x_T, audit [T, L, B] or None, counts)."""
        x, a = self.start(x0, audit)
        for i in range(self.T):
            self.step(i, x, cond, txt, a)
        counts = abi.ff_get_counts(self.ctx)
        return x, (None if a is None else a.view(self.T, self.L, -1)), counts

    def close(self):
        if self.ctx:
            abi.ff_ctx_destroy(self.ctx)
            self.ctx = None
        if self.plan:
            abi.ff_plan_destroy(self.plan)
            self.plan = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def host_inputs_to_device(cfg, inputs, device=_DEV):
    """Seeded host inputs -> device tensors (x fp32, cond fp32, txt in the model dtype or None)."""
    x = torch.from_numpy(np.ascontiguousarray(inputs["x"])).to(device)
    c = torch.from_numpy(np.ascontiguousarray(inputs["c"], dtype=np.float32)).to(device)
    txt = None
    if cfg["n_txt"] > 0:
        txt = torch.from_numpy(np.ascontiguousarray(inputs["txt"], dtype=np.float32)).to(device=device,
                                                                                         dtype=torch_dtype(cfg))
    return x, c, txt
