"""FeatFix cached diffusion-transformer denoising on MI355X (gfx950).

The compute path lives in libfeatfix.so (HIP kernels + C ABI, include/featfix.h);
``abi`` is its ctypes binding and ``pipeline`` keeps weights, cache and workspace in
torch device memory around it.
"""
from . import abi  # noqa: F401

__all__ = ["abi"]
