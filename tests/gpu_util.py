"""Helpers shared by the GPU parity tests (device upload/download, tolerances)."""
import sys

import numpy as np
import torch

import oracle as O
import synth
from paper_2607_27842_amd import abi, pipeline

# Tolerances (normwise max relative error, max|a-b| / max|b|): the accuracy bounds set
# for final latents, reused for block deltas and forecasts.
TOL = {synth.F32: 1e-5, synth.BF16: 2e-2}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def need_gpu():
    assert torch.cuda.is_available(), "GPU test run without a GPU"
    abi.lib()   # fails loudly if libfeatfix.so is missing


def dev(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda").to(dt)


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def tdt(cfg):
    return pipeline.torch_dtype(cfg)


def ulp_close(a, b, dtype):
    """Elementwise agreement within one unit in the last place of the storage dtype
    (values computed in fp32 vs fp64 may round to neighbouring representable values)."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    rel = 2.0 ** -7 if dtype == synth.BF16 else 2.0 ** -21
    scale = np.abs(b).max() + 1e-30
    bad = np.abs(a - b) > rel * np.abs(b) + 1e-6 * scale
    return int(bad.sum())
