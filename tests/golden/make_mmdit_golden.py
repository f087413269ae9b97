#!/usr/bin/env python3
"""Writes the oracle's results for the reduced-depth, full-width MMDiT parity stacks
(synth.reduced_stack: FLUX-like, Qwen-like and HunyuanVideo-like blocks at full width and
token count) to tests/golden/mmdit_<name>_featfix.npz.  It calls only oracle/ and synth/.

The fp64 oracle needs about a minute per FLUX-width block and four per HunyuanVideo-width
block on 8 cores, too slow for a GPU test, so the GPU test reads these files instead.

    python tests/golden/make_mmdit_golden.py [flux qwen hunyuan]

Each file holds the FeatFix loop's final latent x_T (float16: the values are O(1), so the
storage error is below 2^-11 of max|x_T|, which the test subtracts from its tolerance),
max|x_T| in fp64, the per-step, per-layer, per-sample audit (fp64, NaN where no paid check
ran), the counts, the plan arrays, and a JSON record of the workload, the weight options
and the sha256 of the oracle source it came from."""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle as O  # noqa: E402
import synth  # noqa: E402

WEIGHT_OPTS = {"seed": 0, "bias_std": 0.02, "gain_std": 0.1}
ORACLE_SRC = os.path.join(ROOT, "oracle", "featfix_oracle.py")
PLAN_KEYS = ("step_kind", "refresh_ord", "k_eff", "read_slots", "write_slot", "action")
COUNT_KEYS = ("n_full_refresh", "n_paid_checks", "n_forwarded", "n_recomputed")


def path_of(name):
    return os.path.join(HERE, f"mmdit_{name}_featfix.npz")


def oracle_sha():
    return hashlib.sha256(open(ORACLE_SRC, "rb").read()).hexdigest()


def make(name):
    cfg = synth.reduced_stack(name)
    t0 = time.time()
    W = synth.make_weights(cfg, **WEIGHT_OPTS)
    inp = synth.make_inputs(cfg)
    mask = synth.site_mask(cfg)
    print(f"{name}: inputs in {time.time() - t0:.0f}s; running the oracle", flush=True)
    ref = O.run(cfg, O.FEATFIX, inp, W, mask)
    T, L, B = cfg["T"], len(cfg["kinds"]), cfg["B"]
    audit = np.full((T, L, B), np.nan)
    for (i, l), d in ref["audit"].items():
        audit[i, l] = d
    meta = {"workload": cfg, "mode": "featfix", "weights": WEIGHT_OPTS, "inputs": "synth.make_inputs (seeds 1, 2, 3)",
            "oracle_sha256": oracle_sha(), "seconds": round(time.time() - t0, 1)}
    np.savez_compressed(path_of(name), x=ref["x"].astype(np.float16), x_absmax=np.abs(ref["x"]).max(),
                        audit=audit, counts=np.array([ref["counts"][k] for k in COUNT_KEYS], np.int64),
                        meta=np.array(json.dumps(meta)), **{k: np.asarray(ref["plan"][k]) for k in PLAN_KEYS})
    print(f"{name}: wrote {path_of(name)} after {time.time() - t0:.0f}s", flush=True)


if __name__ == "__main__":
    for n in sys.argv[1:] or ["flux", "qwen", "hunyuan"]:
        make(n)
