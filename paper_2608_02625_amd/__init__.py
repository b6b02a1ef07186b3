"""MI355X (gfx950) refinement step of draft-then-refine decoding for diffusion LMs.

One refinement pass: a non-causal transformer forward over prompt+draft, a
fused per-position top-1/confidence reduction over the vocabulary, and the
threshold edit/unmask rule -- all in hand-written HIP kernels behind the C ABI
of include/dlm.h (libdlm.so).  PyTorch supplies device memory and streams.
"""

from ._lib import DlmConfig, DlmError, DlmStats, LIB_PATH, load  # noqa: F401

__all__ = ["DlmConfig", "DlmError", "DlmStats", "LIB_PATH", "load", "Refiner"]


def __getattr__(name):
    if name == "Refiner":
        from .model import Refiner
        return Refiner
    raise AttributeError(name)
