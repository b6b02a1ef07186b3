"""Seeded synthetic workloads for the refinement step.

This package holds only data and seeded input generators: model shapes,
workload sizes, prompt/draft token draws and mask-set draws.  It contains
none of the refinement arithmetic, so both the GPU path's callers and the
CPU oracle may import it.
"""

from .configs import MODELS, WORKLOADS, ModelShape, Workload, model_shape, workload
from .inputs import draw_tokens, draw_mask_set, make_inputs

__all__ = [
    "MODELS", "WORKLOADS", "ModelShape", "Workload", "model_shape", "workload",
    "draw_tokens", "draw_mask_set", "make_inputs",
]
