"""GPU parity of block-AR drafting (Sec. 3.3, Sec. 4.1; b/s/t settings of
Table 9 and Table 10) against the float64 CPU oracle.

Every GPU step is compared with the oracle's step on the same input: top-1
bit-exact where the oracle's top-1/top-2 logit margin exceeds the exemption,
max logits within 2e-2 max-abs-relative, confidences within 2e-2 on their
natural [0, 1] scale (the same tolerance; a probability's reference magnitude
is 1).  The unmasking decision is recomputed by the oracle's
selection rule from the GPU's own float32 confidences and must match bit for
bit; the GPU selection must also equal the oracle's own in every sequence
where no oracle confidence of a masked slot lies within max(1e-2, the
sequence's measured confidence error) of the threshold and the oracle's
confidence gap at the quota cut (a ranking decision) exceeds twice that
error: outside those bands the GPU's confidences are on the oracle's side of
every cut.  The loop entry point must reproduce the step-by-step
trajectory exactly, which also checks the K/V cache it keeps across blocks
(the step entry point recomputes the cache from the tokens every call).
"""

from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_util import HIDDEN_TOL, MARGIN, log, max_abs_rel, need_gpu
from workloads import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu

# Threshold-distance exemption of the parity contract (probability units).
# With the LM head sharpened 10x, logit rounding errors grow 10x and so do
# confidence errors; a sequence whose measured confidence error exceeds this
# band widens it to that error (decisions outside it cannot differ).
CONF_TOL = MARGIN


def _torch():
    import torch
    return torch


def _cuda_i32(a):
    return _torch().tensor(np.ascontiguousarray(a, dtype=np.int32), device="cuda")


def _np(t):
    return t.detach().cpu().numpy()


def _setup(name, **over):
    need_gpu()
    import oracle
    from paper_2608_02625_amd import Refiner
    w = WORKLOADS[name]
    shape = w.model.replace(**over) if over else w.model
    log(f"[draft setup] {name} {over} building model on cuda:0")
    return w, shape, Refiner(shape.as_dict(), w.weight_seed), oracle.OracleWeights(shape, w.weight_seed)


@pytest.fixture(scope="module")
def tiny_sharp():
    return _setup("tiny", lm_head_scale=10.0)


def _prompts(vocab, B, P, seed):
    return np.random.default_rng(seed).integers(0, vocab - 1, size=(B, P)).astype(np.int32)


def _near_cut(conf_ref, conf_err, is_mask, tau, steps_left):
    """True per sequence when an oracle confidence of a masked slot lies within
    max(CONF_TOL, conf_err[b]) of the threshold, or the oracle's confidence
    gap at the selection cut is at most twice the sequence's measured
    confidence error conf_err[b] (only then can the GPU's ranking of the two
    slots differ)."""
    out = []
    for b in range(conf_ref.shape[0]):
        c = np.sort(conf_ref[b][is_mask[b]])[::-1]
        if c.size == 0:
            out.append(False)
            continue
        quota = -(-c.size // steps_left)
        n_sel = max(quota, int(np.sum(c >= tau)))
        near = bool(np.any(np.abs(c - tau) <= max(CONF_TOL, conf_err[b])))
        if 0 < n_sel < c.size:
            near |= bool(c[n_sel - 1] - c[n_sel] <= 2 * conf_err[b])
        out.append(near)
    return np.array(out)


def _check_step(R, W, s, g, P, b, k, steps_left, tau, margin, tag):
    """One GPU step against the oracle's step on the same input; returns
    (tokens before, tokens after, #decisions checked against the oracle)."""
    import oracle
    torch = _torch()
    B, S = g.shape
    tau = float(np.float32(tau))                # the threshold the kernel compares against
    cur = _np(g).copy()
    ref_next, info = oracle.draft_step(W, cur, P, b, k, tau, steps_left)
    c0 = P + k * b
    L = min(b, S - c0)
    t1 = torch.empty(B, L, dtype=torch.int32, device="cuda")
    cf = torch.empty(B, L, dtype=torch.float32, device="cuda")
    stats = torch.zeros(5, dtype=torch.int32, device="cuda")
    ml = torch.empty(B, L, dtype=torch.float32, device="cuda")
    R.draft_step(g, P, b, k, steps_left, tau, top1=t1, conf=cf, stats=stats, max_logit=ml)
    got = _np(g)
    e_ml = max_abs_rel(_np(ml), info["max_logit"])
    assert e_ml <= HIDDEN_TOL, (tag, e_ml)
    gt1, gcf = _np(t1), _np(cf).astype(np.float64)
    is_mask = cur[:, c0:c0 + L] == s.mask_id
    # tokens outside the block untouched
    assert np.array_equal(got[:, :c0], cur[:, :c0]) and np.array_equal(got[:, c0 + L:], cur[:, c0 + L:])
    # reduction parity
    ok = info["margin"] > margin
    assert np.array_equal(gt1[ok], info["top1"][ok]), tag
    conf_err = float(np.max(np.abs(gcf - info["conf"])))
    assert conf_err <= HIDDEN_TOL, (tag, conf_err)
    # the decision from the GPU's own confidences, by the oracle's rule
    sel = oracle.draft_select(is_mask, gcf, tau, steps_left)
    expect = np.where(sel, gt1, cur[:, c0:c0 + L])
    assert np.array_equal(got[:, c0:c0 + L], expect), tag
    # and the oracle's own decision where no confidence sits near the cut
    row_err = np.max(np.abs(gcf - info["conf"]), axis=1)
    near = _near_cut(info["conf"], row_err, is_mask, tau, steps_left)
    rows = ~near
    checked = 0
    if rows.any():
        ok_rows = ok[rows] | ~is_mask[rows]
        assert np.array_equal(sel[rows], info["sel"][rows]), tag
        assert np.array_equal(got[rows, c0:c0 + L][ok_rows], ref_next[rows, c0:c0 + L][ok_rows]), tag
        checked = int(is_mask[rows].sum())
    st = _np(stats).tolist()
    moved = got[:, c0:c0 + L] != cur[:, c0:c0 + L]
    assert st[0] == int(moved.sum()) and st[1] == 0 and st[3] == 1, (tag, st)
    assert st[2] == int(np.sum(got[:, c0:c0 + L] == s.mask_id)), (tag, st)
    log(f"[{tag}] max logit {e_ml:.2e} conf err {conf_err:.2e} unmasked {st[0]} left {st[2]} "
        f"oracle-checked {checked} near-cut rows {int(near.sum())}")
    return cur, got, checked


def _trajectory(R, W, s, prompt, D, b, steps, tau, margin, tag):
    torch = _torch()
    B, P = prompt.shape
    g = _cuda_i32(np.concatenate([prompt, np.full((B, D), s.mask_id, dtype=np.int32)], 1))
    n_blocks = -(-D // b)
    block_steps, checked = [], 0
    for k in range(n_blocks):
        used = 0
        for t in range(steps):
            _, got, c = _check_step(R, W, s, g, P, b, k, steps - t, tau, margin, f"{tag} block {k} step {t}")
            used += 1
            checked += c
            c0 = P + k * b
            if not np.any(got[:, c0:c0 + b] == s.mask_id):
                break
        block_steps.append(used)
    final = _np(g)[:, P:]
    out, st = R.draft(_cuda_i32(prompt) if P else torch.empty(B, 0, dtype=torch.int32, device="cuda"), D, b, steps,
                      tau)
    log(f"[{tag}] block steps {block_steps} loop stats {st}")
    assert np.array_equal(_np(out), final)
    assert st["block_steps"] == block_steps and st["steps_run"] == sum(block_steps)
    assert st["n_masked_left"] == int(np.sum(final == s.mask_id))
    return checked, block_steps


def test_draft_tiny_trajectory(tiny_sharp):
    """Two sequences, prompt 24, 56 draft positions in blocks of 16 (ragged last
    block), 4 steps per block, threshold 0.25 (the draft threshold of Table 10)."""
    w, s, R, W = tiny_sharp
    prompt = _prompts(s.vocab, 2, 24, 7)
    checked, bs = _trajectory(R, W, s, prompt, 56, 16, 4, 0.25, MARGIN * s.lm_head_scale, "tiny draft")
    assert checked > 0
    # threshold above 1: pure quota pacing, every block takes all its steps
    checked2, bs2 = _trajectory(R, W, s, prompt[:1], 40, 16, 4, 2.0, MARGIN * s.lm_head_scale, "tiny quota")
    assert bs2 == [4, 4, 4]


def test_draft_tiny_edge_cases(tiny_sharp):
    """No prompt; a single block longer than the draft; one step per block."""
    w, s, R, W = tiny_sharp
    m = MARGIN * s.lm_head_scale
    _trajectory(R, W, s, np.zeros((1, 0), dtype=np.int32), 32, 16, 3, 0.25, m, "tiny no prompt")
    _trajectory(R, W, s, _prompts(s.vocab, 1, 20, 8), 40, 64, 4, 0.25, m, "tiny one block")
    _, bs = _trajectory(R, W, s, _prompts(s.vocab, 1, 20, 9), 32, 8, 1, 0.875, m, "tiny one step")
    assert bs == [1, 1, 1, 1]


@pytest.fixture(scope="module")
def small():
    return _setup("small_moe")


def test_draft_step_small_moe(small):
    """Mixture-of-experts model, prompt 128, blocks of 64 (Table 10's b64):
    a step on block 2 with blocks 0-1 final and block 2 partly masked (K/V of
    the prompt and two blocks from the caches).  Rows whose top-k router gap
    is within 1e-2 at some layer may route differently and are exempt, as in
    the refinement forward test; at the others max logits within 2e-2, top-1
    exact outside the margin, confidences within 1e-2; decisions as above."""
    import oracle
    torch = _torch()
    w, s, R, W = small
    prompt, draft, _ = make_inputs(w)
    P, b = w.prompt_len, 64
    D = 4 * b
    tok = np.concatenate([prompt, draft[:, :D]], 1).astype(np.int32)
    rng = np.random.default_rng(5)
    c0 = P + 2 * b
    tok[:, c0:c0 + b][rng.random((1, b)) < 0.6] = s.mask_id
    tok[:, c0 + b:] = s.mask_id
    g = _cuda_i32(tok)
    end = c0 + b
    x_ref, infos, _ = oracle.forward(W, tok[:, :end], collect=True,
                                     key_limit=oracle.block_key_limit(P, end, b))
    gap = np.min(np.stack([i["route_gap"] for i in infos]), axis=0)[0, c0:end]
    ref = oracle.lm_head_reduce(W, x_ref[0, c0:end])
    t1 = torch.empty(1, b, dtype=torch.int32, device="cuda")
    cf = torch.empty(1, b, dtype=torch.float32, device="cuda")
    ml = torch.empty(1, b, dtype=torch.float32, device="cuda")
    R.draft_step(g, P, b, 2, 8, 0.875, top1=t1, conf=cf, max_logit=ml)
    gt1, gcf, gml = _np(t1)[0], _np(cf)[0].astype(np.float64), _np(ml)[0]
    keep = gap > MARGIN
    ok = keep & (ref["margin"] > MARGIN)
    e_ml = max_abs_rel(gml[keep], ref["max_logit"][keep])
    e_cf = float(np.max(np.abs(gcf[keep] - ref["conf"][keep])))
    log(f"[small_moe draft step] route-exempt {int((~keep).sum())}/{b}; max logit {e_ml:.2e} "
        f"(all rows {max_abs_rel(gml, ref['max_logit']):.2e}); conf err {e_cf:.2e}; top-1 checked {int(ok.sum())}/{b}")
    assert e_ml <= HIDDEN_TOL
    assert np.array_equal(gt1[ok], ref["top1"][ok])
    assert e_cf <= MARGIN
    is_mask = tok[:, c0:end] == s.mask_id
    sel = oracle.draft_select(is_mask, gcf[None, :], 0.875, 8)
    assert np.array_equal(_np(g)[:, c0:end], np.where(sel, gt1[None, :], tok[:, c0:end]))
    assert np.array_equal(_np(g)[:, :c0], tok[:, :c0])
    # the [MASK] rows enter layer 0 identical, so they share one router gap and
    # are exempt together when it is small; the real-token rows remain
    assert ok.sum() >= b // 4


def test_cascade_tiny(tiny_sharp):
    """Two-model cascade (Sec. 4.3; cost K x T_d + T_r, Sec. 4.2): a one-layer
    drafter (other seed, same vocabulary) drafts, the two-layer refiner refines.
    dlm_cascade equals dlm_draft then dlm_refine_ex bit for bit, with their
    pass counts; the drafter's trajectory agrees with the oracle step by step
    (as above) and the refiner's first pass on the GPU's draft with the
    oracle's pass at non-exempt positions.  Models of different vocabularies
    are refused."""
    import oracle
    from paper_2608_02625_amd import DlmError, Refiner, cascade
    torch = _torch()
    w, s, Rl, Wl = tiny_sharp
    ds = s.replace(n_layers=1)
    Rs, Ws = Refiner(ds.as_dict(), 3), oracle.OracleWeights(ds, 3)
    prompt = _prompts(s.vocab, 2, 24, 11)
    P, D, b, T, td, n_ref, tu, te = 24, 48, 16, 4, 0.25, 4, 0.25, 0.625
    out, st = cascade(Rs, Rl, _cuda_i32(prompt), D, b, T, td, n_ref, tu, te)
    d, dst = Rs.draft(_cuda_i32(prompt), D, b, T, td)
    r = d.clone()
    _, rst = Rl.refine_ex(_cuda_i32(prompt), r, None, n_ref, tu, te)
    log(f"[cascade tiny] {st}")
    assert np.array_equal(_np(out), _np(r))
    assert st["draft_passes"] == dst["steps_run"] == sum(dst["block_steps"])
    assert st["refine_passes"] == rst["steps_run"] and st["refine_stop_reason"] == rst["stop_reason"]
    assert st["draft_ms"] > 0 and st["refine_ms"] > 0
    # the drafter's own trajectory against the oracle
    _trajectory(Rs, Ws, ds, prompt, D, b, T, td, MARGIN * s.lm_head_scale, "cascade drafter")
    # the refiner's first pass on the GPU's draft
    tok = np.concatenate([prompt, _np(d)], 1).astype(np.int32)
    ref_next, info = oracle.refine_step_ex(Wl, tok, P, tu, te)
    g = _cuda_i32(tok)
    cf = torch.empty(tok.shape[0], D, dtype=torch.float32, device="cuda")
    Rl.refine_step_ex(g, P, tu, te, conf=cf)
    thr = np.where(tok[:, P:] == s.mask_id, tu, te)
    row_err = np.max(np.abs(_np(cf) - info["conf"]), axis=1, keepdims=True)
    assert float(row_err.max()) <= HIDDEN_TOL
    ex = (info["margin"] <= MARGIN * s.lm_head_scale) | (np.abs(info["conf"] - thr) <= np.maximum(CONF_TOL, row_err))
    assert np.array_equal(_np(g)[:, P:][~ex], ref_next[:, P:][~ex])
    assert int((~ex).sum()) > 0
    # no refinement passes: the cascade returns the draft
    out0, st0 = cascade(Rs, Rl, _cuda_i32(prompt), D, b, T, td, 0, tu, te)
    assert np.array_equal(_np(out0), _np(d)) and st0["refine_passes"] == 0
    other = Refiner(s.replace(vocab=4096).as_dict(), 0)
    with pytest.raises(DlmError):
        cascade(other, Rl, _cuda_i32(prompt), D, b, T, td, n_ref, tu, te)


@pytest.fixture(scope="module")
def mini():
    need_gpu()
    from paper_2608_02625_amd import Refiner
    w = WORKLOADS["mini_moe"]
    log("[draft mini_moe] building model on cuda:0")
    return w, w.model, Refiner(w.model.as_dict(), w.weight_seed)


def test_draft_mini_moe_properties(mini):
    """The mini-scale MoE workload at full size, in the benchmark's drafting
    configuration (B 8, prompt 256, 384 positions, b64, s16, t0.25), through
    properties that hold at any size: the whole draft is bit-identical run to
    run; drafting 128 positions gives the first two blocks of the 384-position
    draft (later blocks are invisible); with the threshold above 1 every step
    of block 0 unmasks exactly ceil(n / r) slots per sequence; a threshold <= 0
    fills every block in one step; no [MASK] is left."""
    torch = _torch()
    w, s, R = mini
    prompt, _, _ = make_inputs(w)
    B, P, D = w.batch, w.prompt_len, w.draft_len
    pr = _cuda_i32(prompt)
    a, sa = R.draft(pr, D, 64, 16, 0.25)
    b_, sb = R.draft(pr, D, 64, 16, 0.25)
    log(f"[draft mini_moe] {sa}")
    assert np.array_equal(_np(a), _np(b_)) and sa == sb
    assert sa["n_masked_left"] == int((_np(a) == s.mask_id).sum()) == 0
    assert all(1 <= t <= 16 for t in sa["block_steps"]) and sa["steps_run"] == sum(sa["block_steps"])
    short, _ = R.draft(pr, 128, 64, 16, 0.25)
    assert np.array_equal(_np(short), _np(a)[:, :128])
    g = _cuda_i32(np.concatenate([prompt, np.full((B, D), s.mask_id, dtype=np.int32)], 1))
    stats = torch.zeros(5, dtype=torch.int32, device="cuda")
    left = 64
    for t in range(4):
        R.draft_step(g, P, 64, 0, 16 - t, 2.0, stats=stats)
        st = _np(stats).tolist()
        quota = -(-left // (16 - t))
        assert st[0] == B * quota and st[2] == B * (left - quota), (t, st)
        left -= quota
    z, sz = R.draft(pr, D, 64, 16, 0.0)
    log(f"[draft mini_moe] threshold 0: {sz}")
    assert sz["block_steps"] == [1] * 6 and sz["n_masked_left"] == 0


def test_draft_tiny_extreme_blocks(tiny_sharp):
    """Degenerate and maximum block sizes: blocks of one token (causal over the
    response, one step each) and blocks of 1024 (the largest the unmasking
    kernel ranks at once; the second block's window carries 2 x 1024 rows),
    with a ragged last block."""
    w, s, R, W = tiny_sharp
    m = MARGIN * s.lm_head_scale
    _, bs = _trajectory(R, W, s, _prompts(s.vocab, 1, 12, 21), 6, 1, 1, 0.25, m, "tiny block 1")
    assert bs == [1] * 6
    _, bs = _trajectory(R, W, s, _prompts(s.vocab, 1, 16, 22), 1100, 1024, 2, 0.25, m, "tiny block 1024")
    assert len(bs) == 2


def test_cascade_mini_moe_full_size(mini):
    """The benchmark's cascade at full size (mini_drafter drafts B 8 x 384 with
    b64 s16 t0.25, the mini-scale MoE refines up to 4 passes at 0.20): equal
    bit for bit to drafting then refining separately, with the pass counts
    K x T_d + T_r of the two stages."""
    from paper_2608_02625_amd import Refiner, cascade
    from workloads import MODELS
    w, s, R = mini
    Rd = Refiner(MODELS["mini_drafter"].as_dict(), w.weight_seed + 1)
    prompt, _, _ = make_inputs(w)
    pr = _cuda_i32(prompt)
    D = w.draft_len
    out, st = cascade(Rd, R, pr, D, 64, 16, 0.25, 4, 0.2, 0.2)
    d, dst = Rd.draft(pr, D, 64, 16, 0.25)
    r = d.clone()
    _, rst = R.refine_ex(pr, r, None, 4, 0.2, 0.2)
    log(f"[cascade mini_moe] {st}")
    assert np.array_equal(_np(out), _np(r))
    assert st["draft_passes"] == dst["steps_run"] and st["refine_passes"] == rst["steps_run"]
    assert st["draft_passes"] <= 6 * 16 and 1 <= st["refine_passes"] <= 4
    assert int((_np(out) == s.mask_id).sum()) == 0


def test_draft_flash_slice_properties():
    """The flash-scale slice (256 experts top-8, 32 query and 8 key/value heads
    of 128, d 4096) at its benchmark batch (16 x 256 prompt): drafting is
    bit-identical run to run, the 64-position draft is the first block of the
    384-position one, and nothing stays masked."""
    need_gpu()
    from paper_2608_02625_amd import Refiner
    w = WORKLOADS["flash_slice"]
    log("[draft flash_slice] building model on cuda:0")
    R = Refiner(w.model.as_dict(), w.weight_seed)
    prompt, _, _ = make_inputs(w)
    pr = _cuda_i32(prompt)
    a, sa = R.draft(pr, w.draft_len, 64, 16, 0.25)
    b_, sb = R.draft(pr, w.draft_len, 64, 16, 0.25)
    log(f"[draft flash_slice] {sa}")
    assert np.array_equal(_np(a), _np(b_)) and sa == sb
    short, _ = R.draft(pr, 64, 64, 16, 0.25)
    assert np.array_equal(_np(short), _np(a)[:, :64])
    assert sa["n_masked_left"] == 0
    del R


def _dense_case(i):
    rng = np.random.default_rng(3000 + i)
    hd = int(rng.choice([64, 128]))
    while True:
        kv = int(rng.integers(1, 5))
        h = kv * int(rng.integers(1, 4))
        if (h * hd) % 128 == 0 and (kv * hd) % 128 == 0:
            break
    over = dict(n_layers=int(rng.integers(1, 3)), d_model=int(rng.choice([128, 256, 384])), n_heads=h, n_kv_heads=kv,
                head_dim=hd, vocab=int(rng.integers(64, 2000)), ffn_dim=64 * int(rng.integers(1, 9)), n_experts=0,
                top_k=0, expert_ffn_dim=0, n_shared_experts=0, lm_head_scale=10.0)
    B, P = int(rng.integers(1, 4)), int(rng.integers(0, 40))
    b = int(rng.choice([4, 8, 16, 32]))
    D = int(rng.integers(1, 3 * b + 1))
    steps = int(rng.integers(1, 5))
    tau = float(rng.choice([0.25, 0.5, 0.9, 2.0]))
    return over, B, P, D, b, steps, tau, 4000 + i


@pytest.mark.parametrize("i", range(12))
def test_draft_random_dense_shapes(i):
    """Seeded random dense shapes (d_model 128-384, head_dim 64/128, 1-12 query
    heads over 1-4 KV heads, 1-2 blocks, vocabularies of 64-2000, sharpened
    head), ragged batches and block settings (blocks of 4-32, 1-4 steps,
    thresholds 0.25-2.0): every step against the oracle's step on the same
    tokens, and the loop equal to the step-by-step trajectory."""
    need_gpu()
    import oracle
    from paper_2608_02625_amd import Refiner
    over, B, P, D, b, steps, tau, seed = _dense_case(i)
    s = WORKLOADS["tiny"].model.replace(**over)
    R = Refiner(s.as_dict(), seed)
    W = oracle.OracleWeights(s, seed)
    prompt = _prompts(s.vocab, B, P, seed)
    tag = (f"draft sweep {i}: L{s.n_layers} d{s.d_model} H{s.n_heads}/{s.n_kv_heads}x{s.head_dim} F{s.ffn_dim} "
           f"V{s.vocab} B{B} P{P} D{D} b{b} s{steps} t{tau}")
    checked, bs = _trajectory(R, W, s, prompt, D, b, steps, tau, MARGIN * s.lm_head_scale, tag)
    assert len(bs) == -(-D // b) and checked > 0
