#!/usr/bin/env python3
"""Throughput of the FeatFix cached denoising loop on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

A bench step is one denoising step of the FeatFix schedule (time embedding, patch
embedding, every layer's exact block / history refresh / Taylor draft / verify+replace as
the plan says, final layer and Euler update).  Inputs and weights are resident in HBM
before anything is timed.  Workload (value): DiT-XL/2 shape -- 28 DiT blocks, hidden
1152, 16 heads of 72, 256 tokens, batch 8, bf16, T=50, refresh every 5 steps,
second-order forecast, sites at layers 13 and 27 on every cached step.

Timing: W untimed warm-up steps in schedule order; then exactly K steps from step 0 of a
fresh loop, wrapping to a new loop after step T-1 (the window, HIP events around it);
then max(5, ceil(K/T)) whole T-step loops, each timed with its own HIP event pair on the
stream from before step 0 to after step T-1.  value = T / the median loop time (the
steps of a loop differ in cost: refresh steps run every block exactly, cached steps only
the sites, so only whole loops give an unbiased rate).  Verify, Exact-only, Vanilla and
the matched-compute arms are timed the same way, as are the FLUX-like loops; the
Qwen-like and HunyuanVideo-like loops (FeatFix and Vanilla) and a DiT-XL/2 FeatFix loop
with the adaptive (discrepancy-triggered) refresh policy are reported alongside, with a
FLUX-like resolution sweep, a DiT-XL/2 shadow-Vanilla diagnostic, the FLUX-like loop with
rotary embedding and the guided (batch-doubled) DiT-XL/2 loop.

Prints ONE JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "denoise steps/sec at DiT-XL/2 & FLUX-like shape; MFMA util %, HBM GB/s %"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
CALIB_BYTES = 256 << 20     # plain copy of known size, the scale for FETCH_SIZE / WRITE_SIZE
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_gemm_dit_xl2.json")
# the GEMM kernels and the device helpers their epilogue uses: traffic counters belong to these exact sources
# runs of drafted layers applied from per-run history sums formed at the refreshes
# (ff_ctx_hist_sums); --no-hist-sums drafts layer by layer
HIST_SUMS = True
COND_CACHE = True   # conditioning of the whole schedule formed at step 0 (ff_ctx_cond_cache)
GEMM_SOURCES = [os.path.join(ROOT, "paper_2607_27842_amd", "csrc", f) for f in ("k_gemm.hip", "dev_common.h")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def device_inputs(cfg, seed=1):
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    c_lat, F, H, W = cfg["lat"]
    Bx = cfg["B"] // 2 if cfg.get("cfg_pairs") else cfg["B"]     # guided pairs share a latent
    x0 = torch.randn((Bx, c_lat, F, H, W), generator=g, device="cuda", dtype=torch.float32)
    cond = torch.randn((cfg["B"], cfg["C"]), generator=g, device="cuda", dtype=torch.float32)
    txt = None
    dt = torch.bfloat16 if cfg["dtype"] == 1 else torch.float32
    cond = cond.to(dt).float()            # conditioning values are bf16-representable
    if cfg["n_txt"] > 0:
        txt = torch.randn((cfg["B"], cfg["n_txt"], cfg["C"]), generator=g, device="cuda").to(dt)
    return x0, cond, txt


class Loop:
    """Steps through the plan, wrapping to a fresh loop (reset + initial latent) after T-1."""

    def __init__(self, runner, x0, cond, txt):
        import torch
        self.r, self.x0, self.cond, self.txt = runner, x0, cond, txt
        self.x = x0.clone()
        self.audit = torch.full((runner.T * runner.L * runner.dm.cfg["B"],), float("nan"), device="cuda")
        self.pos = 0

    def step(self):
        i = self.pos % self.r.T
        if i == 0:
            from paper_2607_27842_amd import abi
            abi.ff_ctx_reset(self.r.ctx)
            self.x.copy_(self.x0)
        self.r.step(i, self.x, self.cond, self.txt, self.audit)
        self.pos += 1


def timed_steps(loop, n):
    """Exactly n steps from step 0 of a fresh loop (wrapping after T-1), one event pair."""
    import torch
    loop.pos = 0
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(n):
        loop.step()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b)


def time_loops(loop, n):
    """n whole loops, each from step 0 to step T-1 between its own pair of HIP events on
    the stream; returns the loop times in ms."""
    import torch
    T = loop.r.T
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    torch.cuda.synchronize()
    for a, b in ev:
        loop.pos = 0
        a.record()
        for _ in range(T):
            loop.step()
        b.record()
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in ev]


def loop_entry(loop, n_loops):
    """Median whole-loop time and rate of n_loops timed loops, with their spread."""
    import statistics
    ms = time_loops(loop, n_loops)
    med = statistics.median(ms)
    T = loop.r.T
    return {"loops": n_loops, "steps_per_loop": T, "loop_ms_median": round(med, 3),
            "loop_ms_min": round(min(ms), 3), "loop_ms_max": round(max(ms), 3),
            "steps_per_s": round(T / (med / 1e3), 2)}


def per_step_kind_ms(loop):
    """One loop with an event before every step: mean ms of refresh and of cached steps."""
    import torch
    T = loop.r.T
    loop.pos = 0
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(T + 1)]
    torch.cuda.synchronize()
    for i in range(T):
        ev[i].record()
        loop.step()
    ev[T].record()
    torch.cuda.synchronize()
    kinds = loop.r.export_plan()["step_kind"]
    ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(T)]
    ref = [m for m, k in zip(ms, kinds) if k == 0]
    cac = [m for m, k in zip(ms, kinds) if k == 1]
    return sum(ref) / max(1, len(ref)), (sum(cac) / len(cac) if cac else 0.0)


def profile_loop(loop):
    """One whole loop with per-launch HIP events on the same stream (ff_ctx_profile)."""
    import torch
    from paper_2607_27842_amd import abi
    loop.pos = 0
    abi.ff_ctx_profile(loop.r.ctx, 1)
    for _ in range(loop.r.T):
        loop.step()
    torch.cuda.synchronize()
    stats = abi.ff_ctx_profile_read(loop.r.ctx)
    abi.ff_ctx_profile(loop.r.ctx, 0)
    return stats


def calibration_copy():
    """One plain copy kernel of CALIB_BYTES (read) + CALIB_BYTES (write): under rocprofv3
    --pmc its FETCH_SIZE / WRITE_SIZE give the counters' scale for this machine."""
    import torch
    a = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    torch.neg(a, out=b)
    torch.cuda.synchronize()
    del a, b


def gemm_traffic():
    """HBM bytes per GEMM launch measured with rocprofv3 counters for the current GEMM
    source (None if the counters were taken on a different version of the kernel)."""
    import hashlib
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        h.update(open(f, "rb").read())
    sha = h.hexdigest()
    if rec.get("gemm_source_sha256") != sha:
        return None
    return rec.get("bytes_per_launch")


def kernel_table(stats):
    out = {}
    for k, s in stats.items():
        if s["launches"] == 0:
            continue
        sec = s["ms"] / 1e3
        out[k] = {"launches": s["launches"], "avg_us": round(s["ms"] * 1e3 / s["launches"], 3),
                  "total_ms": round(s["ms"], 3),
                  "tflops": round(s["flops"] / sec / 1e12, 1) if s["flops"] else None,
                  "gbs": round(s["bytes"] / sec / 1e9, 1)}
    return out


def adaptive_entry(dm, mask, fixed_loop, x0, cond, txt, n_loops):
    """FeatFix with the adaptive (discrepancy-triggered) refresh policy: tau is the median
    of the fixed-schedule loop's per-step largest site discrepancies (from its last loop's
    audit), so some cached steps trigger a refresh.  Timed like the fixed loop (whole
    loops, median); the time includes the host waits for each checked step's
    discrepancies."""
    import numpy as np
    from paper_2607_27842_amd import abi, pipeline
    r0 = fixed_loop.r
    a = fixed_loop.audit.view(r0.T, r0.L, -1).cpu().numpy()
    per_step = [float(np.nanmax(a[i])) for i in range(r0.T) if np.isfinite(a[i]).any()]
    tau = float(np.median(per_step))
    r = pipeline.Runner(dm, abi.FF_FEATFIX, mask, tau=tau, hist_sums=HIST_SUMS, cond_cache=COND_CACHE)
    loop = Loop(r, x0, cond, txt)
    for _ in range(r.T):
        loop.step()
    entry = {"tau": tau}
    entry.update(loop_entry(loop, n_loops))
    kinds = r.step_kinds()
    entry["counts_per_loop"] = abi.ff_get_counts(r.ctx)
    entry["refresh_steps"] = [i for i, k in enumerate(kinds) if k == abi.FF_STEP_REFRESH]
    log(f"[bench] adaptive featfix (tau {tau:.4g}): {entry['steps_per_s']} steps/s, "
        f"{entry['counts_per_loop']['n_full_refresh']} refreshes per loop")
    r.close()
    return entry


def run_workload(name, mode_names, warmup_steps, n_loops, with_profile, adaptive=False, window_steps=0,
                 loops_for=None, clock=None, per_kind=True):
    """Per mode: warmup_steps untimed steps, the exact window of window_steps steps
    (featfix only, when > 0), n_loops whole timed loops (loops_for[mode] overrides), the
    mean refresh / cached step time of one more loop (per_kind), and (featfix,
    with_profile) one loop with per-launch events."""
    import torch
    import synth
    from paper_2607_27842_amd import abi, pipeline
    cfg = synth.get_config(name)
    t0 = time.time()
    dm = pipeline.DeviceModel.random(cfg, seed=0)
    x0, cond, txt = device_inputs(cfg)
    torch.cuda.synchronize()
    log(f"[bench] {name}: weights on device in {time.time() - t0:.1f}s")
    mask = synth.site_mask(cfg)
    res = {"sites": synth.sites_of(cfg)}
    for mode_name in mode_names:
        mode = synth.MODE_NAMES[mode_name]
        r = pipeline.Runner(dm, mode, mask, hist_sums=HIST_SUMS, cond_cache=COND_CACHE)
        loop = Loop(r, x0, cond, txt)
        for _ in range(warmup_steps):
            loop.step()
        entry = {"warmup_steps": warmup_steps}
        if window_steps and mode_name == "featfix":
            ms = timed_steps(loop, window_steps)
            entry["window"] = {"steps": window_steps, "ms": round(ms, 3),
                               "steps_per_s": round(window_steps / (ms / 1e3), 2)}
        entry.update(loop_entry(loop, (loops_for or {}).get(mode_name, n_loops)))
        if clock and mode_name == "featfix":
            entry["gpu_clock"] = clock.measure(loop)
        ref_ms, cac_ms = per_step_kind_ms(loop) if per_kind else (float("nan"), float("nan"))
        if per_kind:
            entry["ms_refresh_step"] = round(ref_ms, 4)
            entry["ms_cached_step"] = round(cac_ms, 4)
        entry["counts_per_loop"] = abi.ff_get_counts(r.ctx)
        entry["hist_sums"] = r.hsum is not None
        if with_profile and mode_name == "featfix":
            entry["kernels"] = profile_loop(loop)
            entry["plan"] = r.export_plan()
        log(f"[bench] {name} {mode_name}: {entry['steps_per_s']} steps/s over {entry['loops']} loops "
            f"(refresh {ref_ms:.3f} ms, cached {cac_ms:.3f} ms)")
        res[mode_name] = entry
        if adaptive and mode_name == "featfix":
            res["featfix_adaptive"] = adaptive_entry(dm, mask, loop, x0, cond, txt, n_loops)
        r.close()
        del loop, r
    if "featfix" in res and "vanilla" in res:
        res["featfix_over_vanilla"] = round(res["featfix"]["steps_per_s"] / res["vanilla"]["steps_per_s"], 3)
    if "featfix" in res and "verify" in res:
        res["verify_over_featfix_loop_time"] = round(res["verify"]["loop_ms_median"] / res["featfix"]["loop_ms_median"], 4)
    del dm
    torch.cuda.empty_cache()
    return res


def per_layer_draft_profile(name="dit_xl2"):
    """One FeatFix loop drafting layer by layer (no history sums), with per-launch events:
    the HBM rate of the per-layer draft passes under their own byte count."""
    import torch
    import synth
    from paper_2607_27842_amd import pipeline
    cfg = synth.get_config(name)
    dm = pipeline.DeviceModel.random(cfg, seed=0)
    x0, cond, txt = device_inputs(cfg)
    r = pipeline.Runner(dm, synth.MODE_NAMES["featfix"], synth.site_mask(cfg), hist_sums=False, cond_cache=COND_CACHE)
    loop = Loop(r, x0, cond, txt)
    for _ in range(r.T):
        loop.step()
    k = profile_loop(loop)
    r.close()
    del loop, r, dm
    torch.cuda.empty_cache()
    return k


class ClockSampler:
    """The GFX clock of the benchmark's GPU sampled every ~10 ms from a side thread
    (amdsmi) while a timed region runs."""

    def __init__(self):
        self.handle, self.err = None, None
        try:
            import amdsmi
            import torch
            amdsmi.amdsmi_init()
            handles = amdsmi.amdsmi_get_processor_handles()
            bus = getattr(torch.cuda.get_device_properties(0), "pci_bus_id", None)
            pick = handles[0] if len(handles) == 1 else None
            for h in handles:
                bdf = amdsmi.amdsmi_get_gpu_device_bdf(h)
                if bus is not None and int(bdf.split(":")[1], 16) == int(bus):
                    pick = h
            if pick is None:
                raise RuntimeError(f"{len(handles)} GPUs visible to amdsmi and none matched the device's PCI bus")
            self.amdsmi, self.handle = amdsmi, pick
            self.read()
        except Exception as e:   # reported, not fatal: the clock is context for the rates
            self.err = f"{type(e).__name__}: {e}"

    def read(self):
        info = self.amdsmi.amdsmi_get_clock_info(self.handle, self.amdsmi.AmdSmiClkType.GFX)
        return float(info["clk"])

    def measure(self, loop, seconds=3.0):
        """The clock while the loop runs back to back for `seconds` (untimed): the SMU's
        readings refresh every ~0.1 s and lag the load, so the first second's samples are
        dropped and the median of the rest is reported."""
        import statistics
        import threading
        import torch
        if self.handle is None:
            return {"error": self.err}
        samples, run = [], [True]

        def body():
            t0 = time.time()
            while run[0]:
                try:
                    v = self.read()
                except Exception as e:
                    self.err = f"{type(e).__name__}: {e}"
                    return
                if time.time() - t0 > 1.0:
                    samples.append(v)
                time.sleep(0.01)
        th = threading.Thread(target=body, daemon=True)
        th.start()
        t0 = time.time()
        while time.time() - t0 < seconds:
            for _ in range(loop.r.T):
                loop.step()
            torch.cuda.synchronize()
        run[0] = False
        th.join()
        if not samples:
            return {"error": self.err or "no samples"}
        return {"source": f"amdsmi GFX clock sampled every ~10 ms while the FeatFix loop ran back to back for "
                          f"{seconds:.0f} s (first second dropped)",
                "samples": len(samples), "mhz_median": statistics.median(samples),
                "mhz_min": min(samples), "mhz_max": max(samples)}


def shadow_vanilla(name="dit_xl2"):
    """Mechanism diagnostic (synthetic weights): FeatFix and Verify each stepped in lockstep
    with a Vanilla run, every layer's stream compared with Vanilla's (ff_ctx_trace +
    ff_rel_l1, per sample).  Reports the mean distance over the cached steps' layers and
    samples, the distance after the last layer of the last step, and Verify minus FeatFix
    (positive: forwarding lowers the downstream error)."""
    import numpy as np
    import torch
    import synth
    from paper_2607_27842_amd import abi, pipeline
    cfg = synth.get_config(name)
    dm = pipeline.DeviceModel.random(cfg, seed=0)
    x0, cond, txt = device_inputs(cfg)
    mask = synth.site_mask(cfg)
    T, L, B = cfg["T"], len(cfg["kinds"]), cfg["B"]
    E = B * (cfg["n_img"] + cfg["n_txt"]) * cfg["C"]
    dt = pipeline.torch_dtype(cfg)
    out = {}
    van = pipeline.Runner(dm, abi.FF_VANILLA, mask, hist_sums=HIST_SUMS, cond_cache=COND_CACHE)
    vbuf = torch.empty(L * E, dtype=dt, device="cuda")
    van.trace_into(vbuf)
    for mode_name, mode in (("featfix", abi.FF_FEATFIX), ("verify", abi.FF_VERIFY)):
        r = pipeline.Runner(dm, mode, mask, hist_sums=HIST_SUMS, cond_cache=COND_CACHE)
        buf = torch.empty(L * E, dtype=dt, device="cuda")
        r.trace_into(buf)
        xr, _ = r.start(x0, audit=False)
        xv, _ = van.start(x0, audit=False)
        rel = torch.zeros((T, L, B), dtype=torch.float32, device="cuda")
        kinds = r.export_plan()["step_kind"]
        for i in range(T):
            r.step(i, xr, cond, txt)
            van.step(i, xv, cond, txt)
            for l in range(L):
                abi.ff_rel_l1(dm.desc, buf[l * E:].data_ptr(), vbuf[l * E:].data_ptr(), 1e-8, rel[i, l].data_ptr(),
                              r.ws.data_ptr(), r.ws_bytes)
        d = rel.cpu().numpy()
        cached = [i for i in range(T) if kinds[i] == abi.FF_STEP_CACHED]
        out[mode_name] = {"mean_rel_l1_cached_layers": float(d[cached].mean()),
                          "last_step_last_layer": float(d[T - 1, L - 1].mean())}
        r.close()
    van.close()
    out["verify_minus_featfix_mean"] = out["verify"]["mean_rel_l1_cached_layers"] - out["featfix"]["mean_rel_l1_cached_layers"]
    log(f"[bench] shadow vanilla {name}: mean rel-L1 featfix {out['featfix']['mean_rel_l1_cached_layers']:.4g}, "
        f"verify {out['verify']['mean_rel_l1_cached_layers']:.4g}")
    del dm
    torch.cuda.empty_cache()
    return out


def rope_loop():
    """The FLUX-like FeatFix loop with rotary embedding of q and k (axes 16 / 56 / 56 of the
    128 head dims, theta 1e4; text rows at position 0, image rows at their (frame, row,
    column)): one untimed loop, then one timed 50-step loop."""
    import torch
    import synth
    from paper_2607_27842_amd import pipeline
    cfg = synth.get_config("flux", rope_axes=(16, 56, 56), rope_theta=10000.0)
    dm = pipeline.DeviceModel.random(cfg, seed=0)
    x0, cond, txt = device_inputs(cfg)
    r = pipeline.Runner(dm, synth.MODE_NAMES["featfix"], synth.site_mask(cfg), hist_sums=HIST_SUMS, cond_cache=COND_CACHE)
    loop = Loop(r, x0, cond, txt)
    for _ in range(r.T):
        loop.step()
    loop.pos = 0
    ms = timed_steps(loop, r.T)
    r.close()
    del loop, r, dm
    torch.cuda.empty_cache()
    out = {"rope_axes": [16, 56, 56], "steps": cfg["T"], "ms": round(ms, 3), "steps_per_s": round(cfg["T"] / (ms / 1e3), 2)}
    log(f"[bench] flux featfix with rope: {out['steps_per_s']} steps/s")
    return out


def guided_loop(scale=4.0):
    """DiT-XL/2 with classifier-free guidance by batch doubling: 8 guided images, so 16
    model rows (conditional rows 0-7, their unconditional twins 8-15) and one guided Euler
    step per row pair; FeatFix and Vanilla, one untimed loop, then one timed 50-step loop
    each."""
    import torch
    import synth
    from paper_2607_27842_amd import pipeline
    cfg = synth.get_config("dit_xl2", B=16, cfg_pairs=1, cfg_scale=scale)
    dm = pipeline.DeviceModel.random(cfg, seed=0)
    x0, cond, txt = device_inputs(cfg)
    out = {"model_rows": cfg["B"], "images": cfg["B"] // 2, "cfg_scale": scale}
    for mode in ("featfix", "vanilla"):
        r = pipeline.Runner(dm, synth.MODE_NAMES[mode], synth.site_mask(cfg), hist_sums=HIST_SUMS, cond_cache=COND_CACHE)
        loop = Loop(r, x0, cond, txt)
        for _ in range(r.T):
            loop.step()
        loop.pos = 0
        ms = timed_steps(loop, r.T)
        r.close()
        del loop, r
        out[mode] = {"steps": cfg["T"], "ms": round(ms, 3), "steps_per_s": round(cfg["T"] / (ms / 1e3), 2),
                     "images_per_s": round(cfg["B"] // 2 / (ms / 1e3), 2)}
    del dm
    torch.cuda.empty_cache()
    out["featfix_over_vanilla"] = round(out["featfix"]["steps_per_s"] / out["vanilla"]["steps_per_s"], 3)
    log(f"[bench] guided dit_xl2 (16 rows): featfix {out['featfix']['steps_per_s']} steps/s, "
        f"vanilla {out['vanilla']['steps_per_s']} steps/s")
    return out


def resolution_sweep(sides=(512, 768, 1024)):
    """FLUX-like loop latency and peak device memory from 512^2 to 1024^2 images (latent
    side / 8, patch 2: 1024, 2304 and 4096 image tokens + 512 text tokens), FeatFix and
    Vanilla on the same weights: one untimed loop, then one timed 50-step loop each.
    Peak memory is torch's peak allocation over the run of one mode (the shared weights
    included; the previous run's buffers are released first); cache and workspace are
    the library's exact sizes."""
    import torch
    import synth
    from paper_2607_27842_amd import pipeline
    out = []
    for side in sides:
        g = side // 8
        cfg = synth.get_config("flux", lat=(16, 1, g, g), n_img=(side // 16) ** 2)
        dm = pipeline.DeviceModel.random(cfg, seed=0)
        x0, cond, txt = device_inputs(cfg)
        mask = synth.site_mask(cfg)
        row = {"image": f"{side}x{side}", "n_img": cfg["n_img"]}
        for mode_name in ("featfix", "vanilla"):
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
            torch.cuda.reset_peak_memory_stats()
            r = pipeline.Runner(dm, synth.MODE_NAMES[mode_name], mask, hist_sums=HIST_SUMS, cond_cache=COND_CACHE)
            loop = Loop(r, x0, cond, txt)
            for _ in range(r.T):
                loop.step()
            loop.pos = 0
            ms = timed_steps(loop, r.T)
            row[mode_name] = {"s_per_loop": round(ms / 1e3, 4),
                              "peak_gib": round(torch.cuda.max_memory_allocated() / 2**30, 2),
                              "cache_gib": round(r.cache_bytes / 2**30, 3),
                              "workspace_gib": round(r.ws_bytes / 2**30, 3),
                              "hist_sum_gib": round((0 if r.hsum is None else r.hsum.numel()) / 2**30, 3),
                              "cond_cache_gib": round((0 if r.ccache is None else r.ccache.numel()) / 2**30, 3)}
            r.close()
            del loop, r
        row["speedup"] = round(row["vanilla"]["s_per_loop"] / row["featfix"]["s_per_loop"], 3)
        row["featfix_extra_peak_gib"] = round(row["featfix"]["peak_gib"] - row["vanilla"]["peak_gib"], 2)
        log(f"[bench] flux {side}^2: featfix {row['featfix']['s_per_loop']} s, vanilla {row['vanilla']['s_per_loop']} s "
            f"per loop, peak {row['featfix']['peak_gib']} / {row['vanilla']['peak_gib']} GiB")
        out.append(row)
        del dm, x0, cond, txt
        torch.cuda.empty_cache()
    return out


def cpu_baseline(steps=12):
    """The oracle on the host's cores, on a bounded sample of the DiT-XL/2 FeatFix loop:
    the first `steps` steps (refreshes at 0, 5, 10, so cached steps at k_eff = 0, 1 and 2)
    at full depth (28 blocks), width and tokens, for one sample of the batch of 8.
    Samples never interact and exact blocks dominate the oracle's time (drafts are
    elementwise), so the 50-step, batch-8 rate is extrapolated by exact-block count (this
    sample's 3 x 28 + 9 x 2 = 102 against 10 x 28 + 40 x 2 = 360 per loop) and batch, and
    labelled so.  The tiny fp32 workload's whole 10-step loop is timed in every mode, and
    the MMDiT loops are priced per operation (mmdit_cpu_extrapolation)."""
    import oracle as O
    import synth
    cfg = synth.get_config("dit_xl2", T=steps, B=1)
    W = synth.make_weights(cfg)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((i.get("num_threads", 0) for i in threadpool_info()), default=0)
    except Exception:
        blas_threads = 0
    t0 = time.perf_counter()
    ref = O.run(cfg, O.FEATFIX, inp, W, mask)
    dt = time.perf_counter() - t0
    full = synth.get_config("dit_xl2")
    sample_blocks = sum(28 if k == O.REFRESH_STEP else 2 for k in ref["step_kind"])
    R = full["R"]
    loop_blocks = sum(28 if i % R == 0 else 2 for i in range(full["T"]))
    loop_s = dt * (loop_blocks / sample_blocks) * full["B"]
    cores = len(os.sched_getaffinity(0))
    tiny = synth.get_config("tiny")
    Wt = synth.make_weights(tiny)
    it = synth.make_inputs(tiny)
    mt = synth.site_mask(tiny)
    tiny_rates = {}
    for name in ("vanilla", "draft", "verify", "featfix", "exact_only"):
        t1 = time.perf_counter()
        O.run(tiny, synth.MODE_NAMES[name], it, Wt, mt)
        tiny_rates[name] = round(tiny["T"] / (time.perf_counter() - t1), 2)
    return {"value": round(full["T"] / loop_s, 5), "unit": "steps/s", "cores": min(cores, blas_threads or cores),
            "kind": "oracle", "extrapolated": True,
            "sample": f"fp64 NumPy oracle, DiT-XL/2-shaped FeatFix loop: the first {steps} steps (refreshes 0, 5, 10; "
                      f"k_eff up to 2) at full depth, width and tokens for 1 of the 8 samples took {dt:.1f} s "
                      f"({sample_blocks} exact blocks); extrapolated to the 50-step loop by exact-block count "
                      f"({sample_blocks} -> {loop_blocks}) and to batch 8 (samples are independent): "
                      f"{loop_s:.0f} s per loop; host affinity {cores} cores, BLAS threads {blas_threads}",
            "tiny_fp32_steps_per_s": tiny_rates,
            "mmdit_per_block": mmdit_cpu_extrapolation()}


def mmdit_cpu_extrapolation(tokens=256, row_frac=8):
    """The oracle on the host for the MMDiT workloads, per operation, scaled to full size
    and labelled extrapolated: one exact block of each kind at the workload's full width
    over `tokens` rows (a quarter text), scaled to the full token count by the block's
    FLOP count (projections and MLP linear in the tokens, attention quadratic); one draft
    pass (forecast from a two-refresh history, Eq. 2, rounded to bf16) and one verify
    pass (Eq. 4's distance) over 1/row_frac of the rows at full width, scaled linearly
    (both are elementwise), each timed after one untimed pass.  The 50-step FeatFix loop
    is priced from the plan's counts of exact blocks, drafted layers and paid checks.
    Weight values do not change the oracle's time, so the matrices are a small random
    block repeated to shape (fp64, as the oracle computes)."""
    import numpy as np
    import oracle as O
    import synth
    rng = np.random.default_rng(5)
    base = rng.standard_normal(1 << 20) * 0.02

    def fake_set(cfg, kind):
        out = {}
        for name, shp in synth.layer_shapes(cfg, kind).items():
            out[name + "_w"] = np.resize(base, shp)
            out[name + "_b"] = np.zeros((shp[0],))
        if kind != synth.DIT:
            out["q_g"] = np.ones((cfg["d"],))
            out["k_g"] = np.ones((cfg["d"],))
        return out

    def timed(fn):
        fn()
        t0 = time.perf_counter()
        fn()
        return time.perf_counter() - t0

    res = {}
    for name in ("flux", "qwen", "hunyuan"):
        full = synth.get_config(name)
        L, T = len(full["kinds"]), full["T"]
        entry = {"block_s": {}}
        n_txt = min(full["n_txt"], tokens // 4)
        cfg = dict(full, n_txt=n_txt, n_img=tokens - n_txt)
        for kind in sorted(set(full["kinds"])):
            W = {"txt": fake_set(cfg, kind), "img": fake_set(cfg, kind)} if kind == synth.MMDIT_DOUBLE \
                else fake_set(cfg, kind)
            u = rng.standard_normal((1, tokens, cfg["C"]))
            cs = O.silu(rng.standard_normal((1, cfg["C"])))
            t0 = time.perf_counter()
            O.block(kind, u, cs, W, cfg)
            dt = time.perf_counter() - t0
            scale = O.block_flops(full, kind) / O.block_flops(cfg, kind)
            entry["block_s"]["double" if kind == synth.MMDIT_DOUBLE else "single"] = {
                "sample_tokens": tokens, "sample_s": round(dt, 3), "flop_scale": round(scale, 2),
                "full_s": round(dt * scale, 2)}
            del W
        rows = (full["n_img"] + full["n_txt"]) // row_frac
        shp = (1, rows, full["C"])
        cache = O.TaylorCache(full["K"])
        cache.refresh(rng.standard_normal(shp), 0)
        cache.refresh(rng.standard_normal(shp), full["R"])
        u, hf = rng.standard_normal(shp), rng.standard_normal(shp)
        rnd = O.round_bf16 if full["dtype"] == synth.BF16 else (lambda a: a)
        t_draft = timed(lambda: rnd(u + cache.forecast(full["R"] + 1))) * row_frac
        hd = rnd(u + cache.forecast(full["R"] + 1))
        t_verify = timed(lambda: O.rel_l1(hd, hf, full["rel_eps"])) * row_frac
        del cache, u, hd, hf
        plan = O.make_plan(T, L, full["R"], full["K"], full["S"], synth.site_mask(full), O.FEATFIX)
        act = np.asarray(plan["action"])
        kinds = np.asarray(full["kinds"])
        exact = (act == O.EXACT) | (act == O.SITE)
        loop_s = 0.0
        for kind, key in ((synth.MMDIT_DOUBLE, "double"), (synth.MMDIT_SINGLE, "single")):
            if key in entry["block_s"]:
                loop_s += int(exact[:, kinds == kind].sum()) * entry["block_s"][key]["full_s"]
        n_draft, n_check = int((act == O.DRAFT_ACT).sum()), int((act == O.SITE).sum())
        loop_s += (n_draft + n_check) * t_draft + n_check * t_verify
        entry.update({"draft_pass_s": round(t_draft, 3), "verify_pass_s": round(t_verify, 3),
                      "exact_blocks_per_loop": int(exact.sum()), "drafted_layers_per_loop": n_draft,
                      "paid_checks_per_loop": n_check, "loop_s": round(loop_s, 1),
                      "steps_per_s": round(T / loop_s, 6), "extrapolated": True})
        res[name] = entry
        log(f"[bench] CPU oracle {name}: {entry['steps_per_s']} steps/s extrapolated ({loop_s:.0f} s per loop)")
    return res


WORKLOAD_TEXT = {
    "dit_xl2": "DiT-XL/2-shaped FeatFix loop: 28 DiT blocks, hidden 1152, 16x72 heads, MLP 4608, 256 tokens, "
               "batch 8, bf16, T=50, R=5, K=2, S=3, sites {13,27}",
    "flux": "FLUX-like MMDiT FeatFix loop: 19 double + 38 single blocks, hidden 3072, 24x128 heads, MLP 12288, "
            "4096 image + 512 text tokens, batch 1, bf16, T=50, R=6, K=1, S=2, sites {18,37,56}",
}


def hbm_rates(kern, keys=("draft", "verify", "cache")):
    out = {}
    for k in keys:
        s = kern[k]
        if s["launches"]:
            gbs = s["bytes"] / (s["ms"] / 1e3) / 1e9
            out[k] = {"achieved_gbs": round(gbs, 1), "frac": round(gbs / PEAK_HBM_GBS, 4),
                      "avg_launch_us": round(s["ms"] * 1e3 / s["launches"], 3),
                      "bytes_per_launch": s["bytes"] / s["launches"], "launches": s["launches"]}
    return out


def draft_per_layer_accounting(kern, plan, cfg):
    """The loop's drafted layers priced at the per-layer unit of Eq. 2's draft, (k_eff + 3)
    bytes-per-element x E per drafted layer (read u and k_eff + 1 history slots, write the
    draft), over the time of every launch that drafts (the run passes from history sums)
    or feeds them (the history sums formed at refresh steps)."""
    es = 2 if cfg["dtype"] == 1 else 4
    E = cfg["B"] * (cfg["n_img"] + cfg["n_txt"]) * cfg["C"]
    k_eff, action, kinds = plan["k_eff"], plan["action"], plan["step_kind"]
    layers = 0
    nbytes = 0.0
    for i in range(cfg["T"]):
        if kinds[i] != 1:
            continue
        n = int((action[i] == 1).sum())
        layers += n
        nbytes += n * (int(k_eff[i]) + 3) * E * es
    ms = kern["draft"]["ms"] + kern["cache"]["ms"]
    gbs = nbytes / (ms / 1e3) / 1e9
    return {"drafted_layers_per_loop": layers, "per_layer_bytes_per_loop": nbytes,
            "draft_plus_hist_sum_ms_per_loop": round(ms, 4), "effective_gbs": round(gbs, 1),
            "effective_frac": round(gbs / PEAK_HBM_GBS, 4)}


def exact_blocks_only(reps, name="dit_xl2"):
    """Every layer of the workload through ff_block_exact `reps` times and nothing else:
    the loop's exact-block kernels at its shapes, for counter profiles that need few
    dispatches (each layer's fc2 here writes no history slot)."""
    import torch
    import synth
    from paper_2607_27842_amd import abi, pipeline
    cfg = synth.get_config(name)
    dm = pipeline.DeviceModel.random(cfg)
    n = cfg["n_img"] + cfg["n_txt"]
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    u = torch.randn(cfg["B"], n, cfg["C"], device="cuda", generator=g).to(torch.bfloat16)
    h = torch.empty_like(u)
    c = torch.randn(cfg["B"], cfg["C"], device="cuda", generator=g)
    ws_bytes = abi.ff_workspace_bytes(dm.desc)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    for r in range(reps):
        for l in range(len(cfg["kinds"])):
            abi.ff_block_exact(dm.desc, l, dm.lw[l], c.data_ptr(), u.data_ptr(), h.data_ptr(), ws.data_ptr(),
                               ws_bytes, s)
        torch.cuda.synchronize()
        log(f"[bench] exact blocks only: pass {r + 1} of {reps} done")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=250, help="steps of the exact timed window (K)")
    ap.add_argument("--warmup", type=int, default=50, help="untimed warm-up steps (W)")
    ap.add_argument("--no-flux", action="store_true", help="skip the FLUX-like loops reported in extra")
    ap.add_argument("--no-large", action="store_true", help="skip the Qwen-like and HunyuanVideo-like loops")
    ap.add_argument("--no-vanilla", action="store_true")
    ap.add_argument("--no-arms", action="store_true", help="skip the matched-compute arm loops reported in extra")
    ap.add_argument("--no-sweep", action="store_true", help="skip the FLUX-like resolution sweep reported in extra")
    ap.add_argument("--no-guided", action="store_true", help="skip the guided (batch-doubled) DiT-XL/2 loops")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-clock", action="store_true", help="skip the 3 s clock-sampling run (profiling runs)")
    ap.add_argument("--exact-blocks-only", type=int, default=0, metavar="REPS",
                    help="run only the copy calibration and REPS passes of exact blocks (counter profiles)")
    ap.add_argument("--exact-blocks-workload", default="dit_xl2", choices=["dit_xl2", "flux", "qwen", "hunyuan"],
                    help="the workload whose exact blocks --exact-blocks-only runs")
    ap.add_argument("--no-cond-cache", action="store_true",
                    help="form the conditioning (time MLP, modulation) at every step instead of once per loop")
    ap.add_argument("--no-hist-sums", action="store_true",
                    help="apply runs of drafted layers layer by layer instead of from history sums")
    args = ap.parse_args()
    global HIST_SUMS, COND_CACHE
    HIST_SUMS = not args.no_hist_sums
    COND_CACHE = not args.no_cond_cache
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the FeatFix path here is single-GPU "
              "(no sharding or collectives); use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    import synth
    from paper_2607_27842_amd import abi
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    abi.lib()

    calibration_copy()
    if args.exact_blocks_only:
        exact_blocks_only(args.exact_blocks_only, args.exact_blocks_workload)
        return
    clock = None if args.no_clock else ClockSampler()
    name = "dit_xl2"
    cfg = synth.get_config(name)
    T = cfg["T"]
    K, W = args.steps, args.warmup
    n_loops = max(5, -(-K // T))
    modes = ["featfix", "verify", "exact_only"] + ([] if args.no_vanilla else ["vanilla"])
    if not args.no_arms:
        modes += ["tokens_partial", "channels_partial", "recompute"]   # the matched-compute arms
    prim = run_workload(name, modes, W, n_loops, with_profile=True, adaptive=True, window_steps=K, clock=clock)
    ff = prim["featfix"]
    value = ff["steps_per_s"]
    ms_step = 1e3 / value
    kern = ff.pop("kernels")
    plan = ff.pop("plan")
    g = kern["gemm"]
    achieved = g["flops"] / (g["ms"] / 1e3) / 1e12
    roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": gemm_traffic(),
            "kernel": "k_gemm_dl64 / k_gemm_dl / k_gemm_bf16 (all exact-block GEMM launches of one FeatFix loop)",
            "avg_launch_us": round(g["ms"] * 1e3 / g["launches"], 3),
            "flop_per_launch": g["flops"] / g["launches"]}
    hbm = hbm_rates(kern)
    if HIST_SUMS:
        hbm["draft_per_layer_unit"] = draft_per_layer_accounting(kern, plan, cfg)
        hbm["per_layer_path"] = hbm_rates(per_layer_draft_profile(name), ("draft", "verify"))
    extra = {name: prim, "dit_kernels": kernel_table(kern), "hbm_roofline": hbm}
    if not args.no_flux:
        flux = run_workload("flux", ["featfix", "verify", "exact_only"] + ([] if args.no_vanilla else ["vanilla"]),
                            T, 3, with_profile=True, loops_for={"featfix": 5})
        fk = flux["featfix"].pop("kernels")
        flux["featfix"].pop("plan")
        flux["kernels"] = kernel_table(fk)
        flux["hbm_roofline"] = hbm_rates(fk)
        flux["featfix_rope"] = rope_loop()
        extra["flux"] = flux
        if not args.no_sweep:
            extra["flux_resolution_sweep"] = resolution_sweep()
    if not args.no_large:
        for big in ("qwen", "hunyuan"):
            extra[big] = run_workload(big, ["featfix"] + ([] if args.no_vanilla else ["vanilla"]), synth.get_config(big)["T"],
                                      2, with_profile=False, loops_for={"vanilla": 1}, per_kind=False)
    if not args.no_arms:
        extra["dit_xl2_shadow_vanilla"] = shadow_vanilla()
    if not args.no_guided:
        extra["dit_xl2_guided"] = guided_loop()
    out = {"metric": METRIC, "value": round(value, 3), "unit": "steps/s", "n_gpus": 1, "steps": K,
           "warmup": W, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic: seeded N(0,1) latent and class/text vectors, random-init N(0,0.02) weights",
           "config": {"workload": WORKLOAD_TEXT[name] + ("; drafted runs from history sums" if HIST_SUMS
                                                         else "; drafted runs layer by layer")
                                  + ("; conditioning of all steps formed at step 0" if COND_CACHE
                                     else "; conditioning formed at every step"),
                      "global_batch": cfg["B"],
                      "seq_len": cfg["n_img"] + cfg["n_txt"], "parallelism": "none (1 GPU)"},
           "timing": {"value_from": f"median of {n_loops} whole {T}-step loops (HIP events per loop) after {W} "
                                    f"warm-up steps and the {K}-step window",
                      "loops": n_loops, "loop_ms_median": ff["loop_ms_median"], "window": ff.get("window"),
                      "gpu_clock": ff.get("gpu_clock")},
           "roofline": roof}
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle sample ...")
        out["cpu_baseline"] = cpu_baseline()
    out["extra"] = extra
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
