"""CPU oracle for the refinement step -- test infrastructure only.

Plain float64 NumPy (plus a small C weight generator) implementation of one
refinement step and of the refine loop, written from the paper's description
(Sec. 4.2, App. C.4), and of block-AR drafting (Sec. 3.3, Sec. 4.1).  Only tests/, the smoke check and the benchmark's
CPU-baseline leg may import it.  It shares no code with the GPU library.
"""

from .weights import OracleWeights, philox4x32_10, tensor_id  # noqa: F401
from .refine import (  # noqa: F401
    attention, edit_rule, edit_rule_ex, forward, layer_forward, layer_forward_rows, lm_head_reduce, moe_ffn, refine,
    refine_ex, refine_local, refine_step, refine_step_ex,
    rms_norm, rope, route, softmax, swiglu,
)
from .draft import block_key_limit, cascade, draft, draft_forward_block, draft_select, draft_step  # noqa: F401
