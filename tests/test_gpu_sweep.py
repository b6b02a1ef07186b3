"""Seeded sweep of small random model shapes against the oracle.

Each case draws a shape the library accepts (d_model, head_dim 64/128, heads
and KV heads, dense FFN or mixture of experts with top-k and an optional
shared expert, 1-2 blocks, vocabulary size) and a ragged batch (batch 1-3,
prompt 0-80, draft 1-100 tokens, some [MASK] slots).  Per case:

* the full forward against the oracle: for MoE blocks the GPU reports every
  block's router logits and selections; a token routed differently from the
  oracle must be a near-tie (oracle gap within twice that token's measured
  logit error at that block, the rule of R14), and every token routed alike
  at all blocks (every token of a dense model) matches the oracle's hidden
  state within 2e-2 and its top-1 exactly outside the 1e-2 margin;
* the refinement step's top-1 and confidence equal the full forward's bit for
  bit (the step runs the last block's MoE FFN on the draft rows only).
"""

from __future__ import annotations

import os

import numpy as np
import pytest

from tests.gpu_util import HIDDEN_TOL, MARGIN, log, max_abs_rel, need_gpu
from workloads import MODELS
from workloads.inputs import draw_tokens

pytestmark = pytest.mark.gpu

# The committed sweep runs 16 cases; DLM_SWEEP_CASES widens it for a longer
# one-off run (the cases are the same seeded draws, extended).
N_CASES = int(os.environ.get("DLM_SWEEP_CASES", "48"))
# Larger shapes (more K tiles, more experts and tokens per case), fewer of them.
N_BIG = int(os.environ.get("DLM_SWEEP_BIG_CASES", "6"))


def _case(i, big=False):
    rng = np.random.default_rng((5000 if big else 1000) + i)
    hd = int(rng.choice([64, 128]))
    while True:
        kv = int(rng.integers(1, 5))
        h = kv * int(rng.integers(1, 5))
        if (h * hd) % 128 == 0 and (kv * hd) % 128 == 0:
            break
    dims = [768, 1024] if big else [128, 256, 384, 512]
    over = dict(n_layers=int(rng.integers(1, 4 if big else 3)), d_model=int(rng.choice(dims)), n_heads=h,
                n_kv_heads=kv, head_dim=hd, vocab=int(rng.integers(64, 9000 if big else 3000)))
    if rng.random() < 0.7:
        e = int(rng.integers(2, 65 if big else 33))
        over.update(ffn_dim=0, n_experts=e, top_k=int(rng.integers(1, min(8, e) + 1)),
                    expert_ffn_dim=64 * int(rng.integers(1, 9 if big else 5)), n_shared_experts=int(rng.integers(0, 2)))
    else:
        over.update(ffn_dim=64 * int(rng.integers(1, 17 if big else 9)), n_experts=0, top_k=0, expert_ffn_dim=0,
                    n_shared_experts=0)
    if big:
        B, P, D = int(rng.integers(1, 5)), int(rng.integers(0, 201)), int(rng.integers(1, 201))
    else:
        B, P, D = int(rng.integers(1, 4)), int(rng.integers(0, 81)), int(rng.integers(1, 101))
    return MODELS["tiny"].replace(**over), B, P, D, (6000 if big else 2000) + i


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_shape(i):
    _check(*_case(i), f"sweep {i}")


@pytest.mark.parametrize("i", range(N_BIG))
def test_random_larger_shape(i):
    _check(*_case(i, big=True), f"sweep big {i}")


def _check(shape, B, P, D, seed, tag):
    need_gpu()
    import torch
    import oracle
    from paper_2608_02625_amd import Refiner
    R = Refiner(shape.as_dict(), seed)
    W = oracle.OracleWeights(shape, seed)
    rng = np.random.default_rng(seed)
    toks = draw_tokens(rng, (B, P + D), shape.vocab)
    toks[:, P + 1::4] = shape.mask_id
    T, d = toks.size, shape.d_model
    g = torch.tensor(toks, device="cuda")
    out = R.debug_forward(g, P, want_routes=True)
    x_ref, infos, _ = oracle.forward(W, toks, collect=True)
    alike = np.ones(T, dtype=bool)
    n_flip = 0
    if shape.n_experts:
        L, E, k = shape.n_layers, shape.n_experts, shape.top_k
        g_ids = out["routes"].cpu().numpy().reshape(L, T, k)
        g_z = out["router_logits"].cpu().numpy().reshape(L, T, E).astype(np.float64)
        o_z = np.stack([inf["router_logits"].reshape(T, E) for inf in infos])
        o_ids = np.stack([inf["route_ids"].reshape(T, k) for inf in infos])
        gaps = np.stack([inf["route_gap"].reshape(T) for inf in infos])
        err = np.max(np.abs(g_z - o_z), -1)
        assert np.array_equal(np.argsort(-g_z, axis=-1, kind="stable")[..., :k], g_ids)
        differs = np.any(np.sort(g_ids, -1) != np.sort(o_ids, -1), -1)
        assert not np.any(differs & (gaps > 2 * err)), np.argwhere(differs & (gaps > 2 * err))[:4]
        assert max_abs_rel(g_z[0], o_z[0]) <= HIDDEN_TOL       # block 0 reads the exact embeddings
        alike = ~np.any(differs, 0)
        n_flip = int((~alike).sum())
    hid = out["hidden"].cpu().numpy()
    ref = x_ref.reshape(-1, d)
    eh = max_abs_rel(hid[alike], ref[alike]) if alike.any() else 0.0
    red = oracle.lm_head_reduce(W, x_ref[:, P:].reshape(-1, d))
    keep_d = alike.reshape(B, -1)[:, P:].reshape(-1) & (red["margin"] > MARGIN)
    mism = int(np.sum((out["top1"].cpu().numpy() != red["top1"]) & keep_d))
    # the step (last-block MoE FFN on the draft rows) against the full forward
    t1 = torch.empty(B * D, dtype=torch.int32, device="cuda")
    cf = torch.empty(B * D, dtype=torch.float32, device="cuda")
    R.refine_step(g.clone(), P, 1.5, top1=t1, conf=cf)
    torch.cuda.synchronize()
    same = bool(torch.equal(t1, out["top1"]) and torch.equal(cf, out["conf"]))
    log(f"[{tag}] L{shape.n_layers} d{d} H{shape.n_heads}/{shape.n_kv_heads}x{shape.head_dim} "
        f"E{shape.n_experts}k{shape.top_k}F{shape.expert_ffn_dim or shape.ffn_dim}s{shape.n_shared_experts} "
        f"V{shape.vocab} B{B} P{P} D{D}: hidden {eh:.2e} on {int(alike.sum())}/{T} (routing differs for {n_flip}); "
        f"top1 checked {int(keep_d.sum())} mismatches {mism}; step == forward {same}")
    assert eh <= HIDDEN_TOL and mism == 0 and same
