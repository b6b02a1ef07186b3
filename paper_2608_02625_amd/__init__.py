"""MI355X (gfx950) refinement step of draft-then-refine decoding for diffusion LMs.

One refinement pass: a non-causal transformer forward over prompt+draft, a
fused per-position top-1/confidence reduction over the vocabulary, and the
threshold edit/unmask rule -- all in hand-written HIP kernels behind the C ABI
of include/dlm.h (libdlm.so); also block-AR drafting and the two-model
draft-then-refine cascade.  PyTorch supplies device memory and streams.
"""

from ._lib import DlmConfig, DlmError, DlmStats, LIB_PATH, load  # noqa: F401

__all__ = ["DlmConfig", "DlmError", "DlmStats", "LIB_PATH", "load", "Refiner", "cascade"]


def __getattr__(name):
    if name == "Refiner":
        from .model import Refiner
        return Refiner
    if name == "cascade":
        from .model import cascade
        return cascade
    raise AttributeError(name)
