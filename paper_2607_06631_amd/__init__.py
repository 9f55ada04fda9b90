"""Step-pruned video-DiT denoise step for MI355X (gfx950).

The compute lives in libdif.so (hand-written HIP kernels behind the C ABI
of include/dif.h); `binding` marshals torch tensors into it.
"""
from . import flops  # noqa: F401

__all__ = ["binding", "flops"]
