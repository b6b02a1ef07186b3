"""GPU edge cases of the refinement step against the float64 oracle, through
the C ABI: empty expert groups (every token routed to the same k experts;
64 experts for 8 tokens at top-1), sequences of one token (attention over a
single key returns its value), a vocabulary that does not fill the last
256-row tile of the LM head at full model width, and token validation
(ids outside [0, vocab), [MASK] in the prompt: the pass writes nothing and the
synchronising entry points return DLM_ERR_INVALID_ARG)."""

from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_util import HIDDEN_TOL, MARGIN, log, max_abs_rel, need_gpu
from workloads import MODELS
from workloads.inputs import draw_tokens

pytestmark = pytest.mark.gpu

TINY = MODELS["tiny"]


def _np(t):
    return t.detach().cpu().numpy()


def _cuda_i32(a):
    import torch
    return torch.tensor(np.ascontiguousarray(a, dtype=np.int32), device="cuda")


def _models(shape, seed=11):
    need_gpu()
    import oracle
    from paper_2608_02625_amd import Refiner
    return Refiner(shape.as_dict(), seed), oracle.OracleWeights(shape, seed)


def _forward_parity(R, W, toks, P, tag, exempt=None):
    """debug_forward against the oracle: hidden states within 2e-2 on the
    tokens not exempt, top-1 exact outside the margin exemption."""
    import oracle
    shape = W.shape
    out = R.debug_forward(_cuda_i32(toks), P)
    x_ref, infos, _ = oracle.forward(W, toks, collect=True)
    d = shape.d_model
    keep = np.ones(toks.size, dtype=bool) if exempt is None else ~exempt
    eh = max_abs_rel(_np(out["hidden"])[keep], x_ref.reshape(-1, d)[keep])
    red = oracle.lm_head_reduce(W, x_ref[:, P:].reshape(-1, d))
    kd = keep.reshape(toks.shape)[:, P:].reshape(-1) & (red["margin"] > MARGIN)
    mism = int(np.sum((_np(out["top1"]) != red["top1"]) & kd))
    log(f"[{tag}] hidden {eh:.2e} on {int(keep.sum())}/{keep.size} tokens; top1 checked {int(kd.sum())} "
        f"mismatches {mism}")
    assert eh <= HIDDEN_TOL and mism == 0
    return infos


MOE = TINY.replace(d_model=512, n_heads=4, n_kv_heads=1, head_dim=128, ffn_dim=0, n_experts=16, top_k=4,
                   expert_ffn_dim=256, n_shared_experts=1, vocab=2048)


def test_identical_tokens_leave_expert_groups_empty():
    """Every position holds the same token: values are identical at every
    position, so attention returns that value everywhere and all tokens route
    to the same 4 of 16 experts (12 groups empty) in every layer."""
    R, W = _models(MOE)
    B, P, D = 2, 32, 96
    toks = np.full((B, P + D), 555, dtype=np.int32)
    infos = _forward_parity(R, W, toks, P, "identical tokens")
    gaps = np.stack([i["route_gap"] for i in infos])
    assert gaps.min() > MARGIN                            # no routing near-tie anywhere
    import torch
    from oracle.refine import layer_forward
    x = W.embed_rows(toks).astype(np.float64)
    for l in range(MOE.n_layers):
        _, ids = R.debug_layer(l, torch.tensor(x.reshape(B * (P + D), -1), dtype=torch.float32, device="cuda"),
                               B, P + D, want_routes=True)
        sets = {tuple(sorted(r)) for r in _np(ids).tolist()}
        log(f"[identical tokens] layer {l}: GPU expert sets {sets}")
        assert len(sets) == 1
        x, _ = layer_forward(MOE, W.layer(l), x)


def test_top1_of_64_experts_for_8_tokens():
    """64 experts, top-1, 8 tokens: at most 8 groups receive rows."""
    import oracle
    shape = MOE.replace(n_experts=64, top_k=1, expert_ffn_dim=128)
    R, W = _models(shape)
    toks = draw_tokens(np.random.default_rng(4), (1, 8), shape.vocab)
    infos = oracle.forward(W, toks, collect=True)[1]
    near_tie = np.min(np.stack([i["route_gap"] for i in infos]), 0).reshape(-1) <= MARGIN
    _forward_parity(R, W, toks, 4, "64 experts top-1, 8 tokens", exempt=near_tie)
    used = {int(e) for i in infos for e in i["route_ids"].reshape(-1)}
    log(f"[64 experts top-1] experts used by the oracle: {sorted(used)}; near ties {int(near_tie.sum())}")
    assert len(used) <= 2 * 8


@pytest.mark.parametrize("moe", [False, True])
def test_sequence_of_one_token(moe):
    """P = 0, D = 1: each sequence is one token, attention over its single key
    returns its value (the oracle's attention is pinned to that); a batch of
    such sequences must match the oracle, and a refinement pass at threshold
    <= 0 writes each top-1."""
    import torch
    shape = MOE if moe else TINY
    R, W = _models(shape)
    B = 5
    toks = draw_tokens(np.random.default_rng(12), (B, 1), shape.vocab)
    toks[2, 0] = shape.mask_id
    _forward_parity(R, W, toks, 0, f"S=1 {'moe' if moe else 'dense'}")
    g = _cuda_i32(toks)
    t1 = torch.empty(B, dtype=torch.int32, device="cuda")
    st = torch.zeros(5, dtype=torch.int32, device="cuda")
    R.refine_step(g, 0, -1.0, top1=t1, stats=st)
    top = _np(t1).reshape(B, 1)
    assert np.array_equal(_np(g), np.where(top != shape.mask_id, top, toks))
    assert _np(st)[4] == 0


def test_ragged_vocabulary_tile_at_full_width():
    """d_model 2048 with a vocabulary of 150001 ids: the last 256-row tile of
    the LM head holds 241 real rows.  Rows whose normalised hidden state points
    along LM-head rows of that tile put the top-1 there."""
    import torch
    from oracle.refine import lm_head_reduce
    shape = TINY.replace(n_layers=1, d_model=2048, n_heads=16, n_kv_heads=4, head_dim=128, ffn_dim=256,
                         vocab=150001)
    R, W = _models(shape, seed=3)
    B, P, D = 2, 0, 192
    rng = np.random.default_rng(13)
    wlm = W.lm_head()
    tail = np.arange(150001 - 241, 150001)
    targets = rng.choice(tail, size=B * D)
    x = (wlm[targets].astype(np.float64) * 6.0 + rng.standard_normal((B * D, 2048)) * 0.5)
    out = R.debug_head(torch.tensor(x, dtype=torch.float32, device="cuda"), B, P, D)
    rows = np.sort(rng.choice(B * D, size=24, replace=False))
    red = lm_head_reduce(W, x[rows], row_chunk=24)
    ok = red["margin"] > MARGIN
    t1 = _np(out["top1"])[rows]
    em = max_abs_rel(_np(out["max_logit"])[rows], red["max_logit"])
    ec = max_abs_rel(_np(out["conf"])[rows], red["conf"])
    in_tail = int(np.sum(red["top1"] >= tail[0]))
    log(f"[ragged vocab] oracle top-1 in the last tile for {in_tail}/24 rows; checked {int(ok.sum())}; "
        f"max_logit {em:.2e} conf {ec:.2e}")
    assert in_tail >= 12
    assert np.array_equal(t1[ok], red["top1"][ok]) and em <= HIDDEN_TOL and ec <= HIDDEN_TOL
    assert int(_np(out["top1"]).max()) < shape.vocab


def test_invalid_tokens_are_rejected():
    """Ids outside [0, vocab) anywhere, or the [MASK] id in the prompt: a pass
    writes nothing and reports them; dlm_refine and dlm_draft return
    DLM_ERR_INVALID_ARG and leave the caller's draft unchanged."""
    import torch
    from paper_2608_02625_amd import DlmError
    s = TINY
    R, _ = _models(s)
    rng = np.random.default_rng(14)
    B, P, D = 2, 16, 24
    prompt = draw_tokens(rng, (B, P), s.vocab)
    draft = draw_tokens(rng, (B, D), s.vocab)
    cases = {"draft id = vocab": (prompt, np.where(np.arange(D) == 5, s.vocab, draft)),
             "draft id < 0": (prompt, np.where(np.arange(D) == 0, -3, draft)),
             "prompt holds [MASK]": (np.where(np.arange(P) == 2, s.mask_id, prompt), draft),
             "prompt id = vocab + 7": (np.where(np.arange(P) == 15, s.vocab + 7, prompt), draft)}
    for name, (pr, dr) in cases.items():
        d_draft = _cuda_i32(dr)
        with pytest.raises(DlmError, match="outside"):
            R.refine(_cuda_i32(pr), d_draft, None, 4, -1.0)
        assert np.array_equal(_np(d_draft), dr), name
        tok = np.concatenate([pr, dr], 1).astype(np.int32)
        g = _cuda_i32(tok)
        st = torch.zeros(5, dtype=torch.int32, device="cuda")
        R.refine_step(g, P, -1.0, stats=st)
        stats = _np(st).tolist()
        log(f"[invalid tokens] {name}: refine_step stats {stats}")
        n_bad = int(np.sum((tok < 0) | (tok >= s.vocab)) + np.sum(tok[:, :P] == s.mask_id))
        assert stats[4] == n_bad and stats[0] == stats[1] == 0 and np.array_equal(_np(g), tok), name
    # a valid call on the same workspace afterwards runs normally
    d_draft = _cuda_i32(draft)
    _, st = R.refine(_cuda_i32(prompt), d_draft, None, 2, -1.0)
    assert st["n_invalid"] == 0 and st["steps_run"] >= 1
    # drafting: a [MASK] id in the prompt, and an out-of-range id in a block
    with pytest.raises(DlmError, match="outside"):
        R.draft(_cuda_i32(np.where(np.arange(P) == 0, s.mask_id, prompt)), D, 8, 2, 0.5)
    tok = np.concatenate([prompt, np.full((B, D), s.mask_id, dtype=np.int32)], 1)
    tok[1, P + 3] = s.vocab
    g = _cuda_i32(tok)
    st = torch.zeros(5, dtype=torch.int32, device="cuda")
    R.draft_step(g, P, 8, 0, 2, 0.0, stats=st)
    assert _np(st)[4] == 1 and np.array_equal(_np(g), tok)


def test_step_draft_rows_equal_full_forward_moe():
    """The step's last-block MoE FFN on the draft rows alone gives the same
    top-1 tokens and confidences, bit for bit, as the full forward, also with
    a prompt that is not a multiple of the router's 32-token groups."""
    import torch
    R, _ = _models(MOE)
    rng = np.random.default_rng(5)
    B, P, D = 3, 37, 45
    toks = draw_tokens(rng, (B, P + D), MOE.vocab, "uniform").astype(np.int32)
    toks[:, P + 3::7] = MOE.mask_id
    g = _cuda_i32(toks)
    out = R.debug_forward(g, P)
    t1 = torch.empty(B * D, dtype=torch.int32, device="cuda")
    cf = torch.empty(B * D, dtype=torch.float32, device="cuda")
    R.refine_step(g.clone(), P, 1.5, top1=t1, conf=cf)
    torch.cuda.synchronize()
    assert torch.equal(t1, out["top1"]) and torch.equal(cf, out["conf"])

