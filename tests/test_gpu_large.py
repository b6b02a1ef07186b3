"""GPU parity at the two largest workloads, run at full size in the launch
configuration of the benchmark and checked on sampled outputs:

  * mini-scale MoE at batch 32 x (256 + 768) tokens with Zipf(1.1) tokens and
    a complete draft (expert load imbalance);
  * the flash-scale layer slice (d 4096, 32 heads, 256 experts of width 1536)
    at batch 16 x (256 + 384).

The float64 oracle evaluates one block only at sampled positions of one
sequence (keys and values from the whole sequence), the GPU runs the block on
the whole batch; the LM head is compared on sampled draft rows; properties
that hold at any size are checked on the whole refinement pass.
"""

from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_util import HIDDEN_TOL, MARGIN, log, max_abs_rel, need_gpu
from workloads import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu

LARGE = ["mini_moe_b32_zipf", "flash_slice"]


def _np(t):
    return t.detach().cpu().numpy()


@pytest.fixture(scope="module", params=LARGE)
def large(request):
    need_gpu()
    import torch
    import oracle
    from paper_2608_02625_amd import Refiner
    w = WORKLOADS[request.param]
    log(f"[{w.name}] building the refiner on cuda:0")
    R = Refiner(w.model.as_dict(), w.weight_seed)
    W = oracle.OracleWeights(w.model, w.weight_seed, cache_layers=False)
    prompt, draft, mask = make_inputs(w)
    toks = np.concatenate([prompt, np.where(mask, w.model.mask_id, draft)], 1).astype(np.int32)
    torch.cuda.synchronize()
    yield w, R, W, toks
    del R
    torch.cuda.empty_cache()


def test_weights_sampled_bit_exact_large(large):
    from oracle import weights as ow
    from tests.test_gpu_mini import _gpu_values
    w, R, W, _ = large
    s = w.model
    d, F, V, E = s.d_model, s.expert_ffn_dim, s.vocab, s.n_experts
    rng = np.random.default_rng(6)
    f = s.n_layers
    cases = [(0, ow.K_EMBED, 0, V, d), (0, ow.K_LM_HEAD, 0, V, d),
             (f, ow.K_WK, 0, s.n_kv_heads * s.head_dim, d), (f, ow.K_ROUTER, 0, E, d),
             (f, ow.K_EXP_GATE, E - 1, F, d), (f, ow.K_EXP_DOWN, E // 2, d, F), (1, ow.K_SH_UP, 0, F, d)]
    for (lf, kind, e, rows, cols) in cases:
        idx = rng.integers(0, rows * cols, size=2048).astype(np.int64)
        got = _gpu_values(R, lf, kind, e, idx, cols, rows)
        ref = ow.weight_values_at(W.seed, ow.tensor_id(lf, kind, e), idx.astype(np.uint64), s.init_std)
        assert np.array_equal(got, ref), (lf, kind, e)


def test_layer0_sampled_rows_large(large):
    """Block 0 on the embedded workload tokens: GPU on the whole batch, the
    oracle at 8 sampled positions of sequence 0; routing checked token by
    token as in the mini-scale test, hidden states on the positions routed
    alike."""
    import torch
    from oracle.refine import layer_forward_rows
    from tests.test_gpu_mini import check_routing
    w, R, W, toks = large
    s = w.model
    B, S, d = w.batch, w.seq_len, s.d_model
    x_in = W.embed_rows(toks).astype(np.float32)                       # [B, S, d]
    xg = torch.tensor(x_in.reshape(B * S, d), device="cuda")
    y, ids, z = R.debug_layer(0, xg, B, S, want_router_logits=True)
    rows = np.sort(np.random.default_rng(8).choice(S, size=8, replace=False))
    log(f"[{w.name} layer 0] oracle block at {len(rows)} positions of sequence 0")
    ref, info = layer_forward_rows(s, W.layer(0), x_in[0].astype(np.float64), rows)
    got = _np(y).reshape(B, S, d)[0, rows]
    gids = _np(ids).reshape(B, S, -1)[0, rows]
    gz = _np(z).reshape(B, S, -1)[0, rows]
    same = check_routing(gids, gz, info["route_ids"], info["router_logits"], info["route_gap"],
                         f"{w.name} layer 0")
    err = max_abs_rel(got[same], ref[same]) if same.any() else 0.0
    log(f"[{w.name} layer 0] hidden max-abs-rel {err:.2e} on {int(same.sum())}/{len(rows)} positions routed alike")
    assert same.any() and err <= HIDDEN_TOL


def test_head_sampled_rows_large(large):
    import torch
    from oracle.refine import lm_head_reduce
    w, R, W, toks = large
    s = w.model
    B, P, D, d = w.batch, w.prompt_len, w.draft_len, s.d_model
    rng = np.random.default_rng(9)
    x = (rng.standard_normal((B, w.seq_len, d)) * 0.5 + W.embed_rows(toks) * 20.0).astype(np.float32)
    out = R.debug_head(torch.tensor(x.reshape(-1, d), device="cuda"), B, P, D)
    rows = np.sort(rng.choice(B * D, size=32, replace=False))
    xr = x[:, P:, :].reshape(B * D, d)[rows].astype(np.float64)
    log(f"[{w.name} head] oracle reduction over {len(rows)} rows x {s.vocab} vocabulary")
    red = lm_head_reduce(W, xr, row_chunk=32)
    ok = red["margin"] > MARGIN
    mism = int(np.sum((_np(out["top1"])[rows] != red["top1"]) & ok))
    em = max_abs_rel(_np(out["max_logit"])[rows], red["max_logit"])
    ec = max_abs_rel(_np(out["conf"])[rows], red["conf"])
    log(f"[{w.name} head] top1 checked {int(ok.sum())}/{len(rows)} mismatches {mism}; "
        f"max_logit {em:.2e}; conf {ec:.2e}")
    assert mism == 0 and em <= HIDDEN_TOL and ec <= HIDDEN_TOL


def test_step_properties_large(large):
    """Threshold above 1 changes nothing; threshold <= 0 writes every
    non-[MASK] top-1; two passes agree bit for bit."""
    import torch
    w, R, W, toks = large
    s = w.model
    B, P, D = w.batch, w.prompt_len, w.draft_len
    t0 = torch.tensor(toks, device="cuda")
    g = t0.clone()
    st = torch.zeros(5, dtype=torch.int32, device="cuda")
    R.refine_step(g, P, 1.5, stats=st)
    assert torch.equal(g, t0) and _np(st)[:2].tolist() == [0, 0]
    outs = []
    for _ in range(2):
        g2 = t0.clone()
        t1 = torch.empty(B * D, dtype=torch.int32, device="cuda")
        cf = torch.empty(B * D, dtype=torch.float32, device="cuda")
        R.refine_step(g2, P, -1.0, top1=t1, conf=cf)
        outs.append((g2, t1, cf))
    assert all(torch.equal(a, b) for a, b in zip(outs[0], outs[1]))
    g2, t1, _ = outs[0]
    top = _np(t1).reshape(B, D)
    new = _np(g2)
    assert np.array_equal(new[:, :P], toks[:, :P])
    assert np.array_equal(new[:, P:], np.where(top != s.mask_id, top, toks[:, P:]))
    log(f"[{w.name} step] tau=-1 changed {int((new != toks).sum())} of {B * D} draft slots")
