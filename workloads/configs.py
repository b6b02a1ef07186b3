"""Model shapes and workloads for the refinement step.

The refiner is a non-causal (bidirectional) pre-norm transformer whose forward
pass runs over the whole prompt+response sequence (Sec. 4.2); the paper does not
describe the refiner's internals, so the shapes below are synthetic
mixture-of-experts diffusion-LM stand-ins sized like the small ("mini") and
large ("flash") models it composes (Sec. 4.3, Sec. 5.1).  Response budgets of
384 tokens follow the paper's generation-length suffixes (Sec. 5.2) and its
refine setting of a 384-token span (Table 10).

Every field here is plain data.  The weight values themselves are produced from
a seed by a counter-based generator that each side (GPU library, CPU oracle)
implements on its own.
"""

from __future__ import annotations

import dataclasses
from dataclasses import dataclass


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int            # dense SwiGLU width (used when n_experts == 0)
    n_experts: int          # routed experts (0 = dense FFN)
    top_k: int
    expert_ffn_dim: int     # routed and shared expert SwiGLU width
    n_shared_experts: int   # 0 or 1
    vocab: int
    rope_theta: float = 10000.0
    norm_eps: float = 1e-6
    init_std: float = 0.02
    lm_head_scale: float = 1.0

    @property
    def mask_id(self) -> int:
        # The last vocabulary id is reserved as [MASK]; token draws never
        # produce it.
        return self.vocab - 1

    @property
    def is_moe(self) -> bool:
        return self.n_experts > 0

    def replace(self, **kw) -> "ModelShape":
        return dataclasses.replace(self, **kw)

    def as_dict(self) -> dict:
        d = dataclasses.asdict(self)
        d["mask_id"] = self.mask_id
        return d


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    batch: int
    prompt_len: int
    draft_len: int
    mask_frac: float        # fraction of draft positions placed in the mask set
    threshold: float        # confidence threshold of the edit/unmask rule
    n_steps: int            # refinement step budget (an upper bound)
    token_dist: str         # "uniform" or "zipf1.1"
    weight_seed: int
    input_seed: int

    @property
    def seq_len(self) -> int:
        return self.prompt_len + self.draft_len

    @property
    def tokens(self) -> int:
        return self.batch * self.seq_len

    @property
    def refined_positions(self) -> int:
        return self.batch * self.draft_len


MODELS = {
    # Tiny dense bidirectional model: 2 layers, d 256, 4 heads of 64, SwiGLU 1024.
    "tiny": ModelShape(n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
                       ffn_dim=1024, n_experts=0, top_k=0, expert_ffn_dim=0,
                       n_shared_experts=0, vocab=2048),
    # Small MoE: 4 layers, d 1024, 16 heads of 64, 32 experts top-4 (width 512) + 1 shared.
    "small_moe": ModelShape(n_layers=4, d_model=1024, n_heads=16, n_kv_heads=16, head_dim=64,
                            ffn_dim=0, n_experts=32, top_k=4, expert_ffn_dim=512,
                            n_shared_experts=1, vocab=32768),
    # Mini-scale MoE: 20 layers, d 2048, 16 heads of 128 with 4 KV heads,
    # 64 experts top-8 (width 1024) + 1 shared, 157184-token vocabulary.
    "mini_moe": ModelShape(n_layers=20, d_model=2048, n_heads=16, n_kv_heads=4, head_dim=128,
                           ffn_dim=0, n_experts=64, top_k=8, expert_ffn_dim=1024,
                           n_shared_experts=1, vocab=157184),
    # Drafter for the two-model cascade with mini_moe as refiner (same
    # 157184-token vocabulary): 8 layers, d 1024, 16 heads of 64 with 4 KV
    # heads, 32 experts top-4 (width 512) + 1 shared.
    "mini_drafter": ModelShape(n_layers=8, d_model=1024, n_heads=16, n_kv_heads=4, head_dim=64,
                               ffn_dim=0, n_experts=32, top_k=4, expert_ffn_dim=512,
                               n_shared_experts=1, vocab=157184),
    # Flash-scale 8-layer slice: d 4096, 32 heads of 128 with 8 KV heads,
    # 256 experts top-8 (width 1536) + 1 shared.
    "flash_slice": ModelShape(n_layers=8, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                              ffn_dim=0, n_experts=256, top_k=8, expert_ffn_dim=1536,
                              n_shared_experts=1, vocab=157184),
}

WORKLOADS = {
    "tiny": Workload("tiny", MODELS["tiny"], batch=1, prompt_len=64, draft_len=64,
                     mask_frac=0.30, threshold=0.9, n_steps=4, token_dist="uniform",
                     weight_seed=0, input_seed=1),
    "small_moe": Workload("small_moe", MODELS["small_moe"], batch=1, prompt_len=128,
                          draft_len=384, mask_frac=0.20, threshold=0.9, n_steps=8,
                          token_dist="uniform", weight_seed=0, input_seed=1),
    "mini_moe": Workload("mini_moe", MODELS["mini_moe"], batch=8, prompt_len=256,
                         draft_len=384, mask_frac=0.10, threshold=0.8, n_steps=4,
                         token_dist="uniform", weight_seed=0, input_seed=1),
    "mini_moe_b32_zipf": Workload("mini_moe_b32_zipf", MODELS["mini_moe"], batch=32,
                                  prompt_len=256, draft_len=768, mask_frac=0.0,
                                  threshold=0.95, n_steps=2, token_dist="zipf1.1",
                                  weight_seed=0, input_seed=2),
    "flash_slice": Workload("flash_slice", MODELS["flash_slice"], batch=16, prompt_len=256,
                            draft_len=384, mask_frac=0.10, threshold=0.8, n_steps=2,
                            token_dist="uniform", weight_seed=0, input_seed=3),
}


def model_shape(name: str) -> ModelShape:
    return MODELS[name]


def workload(name: str) -> Workload:
    return WORKLOADS[name]
