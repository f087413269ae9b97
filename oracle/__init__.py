"""CPU oracle of the FeatFix cached denoising loop -- TEST INFRASTRUCTURE ONLY.

Plain, slow NumPy code in fp64 that states what the GPU path must compute.  Only the
tests, the `__graft_entry__.smoke()` check and the benchmark's CPU-baseline leg may import it; the
product path (the C-ABI library and its Python binding) never does, and this package
imports nothing from the product.

Every function here is pinned by a CPU test against something other than itself
(closed forms, brute force, library routines, invariants the paper states); the only
part without an external pin is the whole-loop latent for random weights, which is
"parity unpinned" against the paper (the paper prints no worked example).
"""
from .featfix_oracle import *  # noqa: F401,F403
