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


# Audit (Eq. 4 discrepancy) tolerance.  fp32: absolute, at the latent's bound.  bf16: relative
# to the oracle's value.  The GPU and the oracle round h_f and h_d to bf16 at the same
# points, from unrounded values that differ by fp32-vs-fp64 accumulation; a one-ulp flip
# of an element moves its |h_d - h_f| by at most 2^-8 |h_f|, and the flips have no
# preferred sign, so the sums Sum|h_d - h_f| and Sum|h_f| over a sample's N*C elements
# move by far less than 2 % of themselves.
AUDIT_RTOL = {synth.F32: 0.0, synth.BF16: 2e-2}
AUDIT_ATOL = {synth.F32: 1e-5, synth.BF16: 1e-4}


def check_audit(a, ref_audit, dtype, idx=None, label="", atol=None):
    """GPU audit a [T, L, B] (numpy) against the oracle's {(i, l): d[B]}; idx selects the
    GPU's samples that the oracle followed.  Returns the largest relative deviation."""
    worst = 0.0
    for (i, l), d in ref_audit.items():
        g = a[i, l] if idx is None else a[i, l][idx]
        np.testing.assert_allclose(g, d, rtol=AUDIT_RTOL[dtype], atol=AUDIT_ATOL[dtype] if atol is None else atol,
                                   err_msg=f"audit step {i} layer {l}")
        worst = max(worst, float(np.max(np.abs(g - d) / np.maximum(np.abs(d), 1e-30))))
    say(f"  {label}audit: {len(ref_audit)} paid checks, largest relative deviation {worst:.3e}")
    return worst
