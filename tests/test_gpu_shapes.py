"""Forward parity on small synthetic shapes that cover what the named workloads
do not all cover at once: grouped-query attention, head_dim 128, batch > 1,
sequence lengths that are not multiples of the 64/128-wide tiles, a one-token
draft, MoE with top-k = E and without a shared expert."""

from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_util import HIDDEN_TOL, MARGIN, log, max_abs_rel, need_gpu
from workloads import MODELS
from workloads.inputs import draw_tokens

pytestmark = pytest.mark.gpu

BASE = MODELS["tiny"]

SHAPES = {
    # name: (shape overrides, batch, prompt_len, draft_len)
    "gqa_hd128_b2": (dict(d_model=512, n_heads=8, n_kv_heads=2, head_dim=128, ffn_dim=1024, vocab=4096), 2, 64, 192),
    "gqa_hd64_ragged": (dict(d_model=256, n_heads=8, n_kv_heads=2, head_dim=64, ffn_dim=512, vocab=1000), 3, 37, 100),
    "mha_hd128_short": (dict(d_model=256, n_heads=2, n_kv_heads=2, head_dim=128, ffn_dim=256, vocab=640), 2, 5, 1),
    # >= 4096 tokens: the QKV and O projections switch to 256-row tiles
    "gqa_hd128_4k_tokens": (dict(d_model=512, n_heads=4, n_kv_heads=2, head_dim=128, ffn_dim=512, vocab=1024), 8, 200, 320),
    "moe_gqa_hd128": (dict(d_model=512, n_heads=4, n_kv_heads=1, head_dim=128, ffn_dim=0, n_experts=16, top_k=4,
                           expert_ffn_dim=256, n_shared_experts=1, vocab=2048), 2, 96, 160),
    "moe_k_eq_e_noshared": (dict(d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, ffn_dim=0, n_experts=4, top_k=4,
                                 expert_ffn_dim=128, n_shared_experts=0, vocab=512), 2, 30, 70),
}


@pytest.mark.parametrize("name", list(SHAPES))
def test_forward_shape(name):
    need_gpu()
    import torch
    import oracle
    from paper_2608_02625_amd import Refiner
    over, B, P, D = SHAPES[name]
    shape = BASE.replace(**over)
    R = Refiner(shape.as_dict(), 11)
    W = oracle.OracleWeights(shape, 11)
    rng = np.random.default_rng(3)
    toks = draw_tokens(rng, (B, P + D), shape.vocab)
    toks[:, P::3] = shape.mask_id                       # some [MASK] slots in the draft
    out = R.debug_forward(torch.tensor(toks, device="cuda"), P)
    x_ref, infos, _ = oracle.forward(W, toks, collect=True)
    d = shape.d_model
    if shape.n_experts and shape.top_k < shape.n_experts:
        gap = np.min(np.stack([i["route_gap"] for i in infos]), axis=0).reshape(-1)
        keep = gap > MARGIN
    else:
        keep = np.ones(B * (P + D), dtype=bool)
    hid = out["hidden"].cpu().numpy()
    eh = max_abs_rel(hid[keep], x_ref.reshape(-1, d)[keep])
    red = oracle.lm_head_reduce(W, x_ref[:, P:].reshape(-1, d))
    keep_d = keep.reshape(B, -1)[:, P:].reshape(-1) & (red["margin"] > MARGIN)
    mism = int(np.sum((out["top1"].cpu().numpy() != red["top1"]) & keep_d))
    em = max_abs_rel(out["max_logit"].cpu().numpy()[keep_d], red["max_logit"][keep_d]) if keep_d.any() else 0.0
    log(f"[{name}] hidden {eh:.2e} on {int(keep.sum())}/{keep.size} tokens; max_logit {em:.2e}; "
        f"top1 checked {int(keep_d.sum())} mismatches {mism}")
    assert eh <= HIDDEN_TOL and em <= HIDDEN_TOL and mism == 0
