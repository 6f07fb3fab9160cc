"""MI355X (gfx950) hot path of ADEPT's token-level early-exit forward pass.

libadept.so (HIP kernels behind the C ABI of include/adept.h) does all the
arithmetic; `binding` marshals torch tensors into it and `model` drives the
layer loop.  Build with `python -m paper_2601_03700_amd.build`.
"""
from . import binding  # noqa: F401

__all__ = ["binding", "model"]
