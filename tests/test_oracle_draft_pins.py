"""Pins of the block-AR drafting oracle (Sec. 3.3, Sec. 4.1; b/s/t settings of
Table 9 and Table 10) against values fixed by hand, by the mathematics and by
independent library routines."""

from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from oracle.draft import block_key_limit, draft, draft_forward_block, draft_select, draft_step
from oracle.refine import attention, forward, lm_head_reduce
from workloads import WORKLOADS, make_inputs


def test_block_key_limit_by_hand():
    # prompt 3, blocks of 2 over 5 draft positions (last block ragged)
    assert block_key_limit(3, 8, 2).tolist() == [3, 3, 3, 5, 5, 7, 7, 8]
    # no prompt, one block covering everything: plain bidirectional
    assert block_key_limit(0, 5, 5).tolist() == [5] * 5
    assert block_key_limit(0, 5, 8).tolist() == [5] * 5
    # block of one: causal over the response, prompt bidirectional
    assert block_key_limit(2, 5, 1).tolist() == [2, 2, 3, 4, 5]


def test_attention_key_limit_against_sdpa_mask():
    """The limited attention equals torch's SDPA with the explicit boolean
    mask; a limit of 1 returns v[0]; limits = S give the unmasked result."""
    rng = np.random.default_rng(11)
    S, H, KV, hd = 19, 4, 2, 16
    q = rng.standard_normal((S, H, hd))
    k = rng.standard_normal((S, KV, hd))
    v = rng.standard_normal((S, KV, hd))
    lim = block_key_limit(5, S, 4)
    o = attention(q, k, v, lim)
    mask = torch.from_numpy(np.arange(S)[None, :] < lim[:, None])
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(np.repeat(k, H // KV, axis=1)).permute(1, 0, 2)
    tv = torch.from_numpy(np.repeat(v, H // KV, axis=1)).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask)
    np.testing.assert_allclose(o, ref.permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-13)
    one = attention(q, k, v, np.ones(S, dtype=int))
    assert np.allclose(one, np.repeat(v[:1], H // KV, axis=1).repeat(S, axis=0), rtol=1e-15)
    np.testing.assert_allclose(attention(q, k, v, np.full(S, S)), attention(q, k, v), rtol=0, atol=0)


@pytest.fixture(scope="module")
def tiny():
    w = WORKLOADS["tiny"]
    return w, oracle.OracleWeights(w.model, w.weight_seed)


def test_block_causal_forward(tiny):
    """Prompt rows equal the forward of the prompt alone; rows of blocks <= j do
    not move when a later block changes; a change inside block j reaches its
    first row (bidirectional within the block); with no prompt and one block
    the mask is no mask."""
    w, W = tiny
    prompt, draft_, _ = make_inputs(w)
    P, b = 16, 8
    t = np.concatenate([prompt[:, :P], draft_[:, :4 * b]], 1)
    S = t.shape[1]
    lim = block_key_limit(P, S, b)
    x = forward(W, t, key_limit=lim)
    np.testing.assert_allclose(x[:, :P], forward(W, t[:, :P]), rtol=0, atol=1e-12)
    t2 = t.copy()
    t2[0, P + 2 * b + 3] = (t2[0, P + 2 * b + 3] + 5) % (w.model.vocab - 1)     # a token of block 2
    x2 = forward(W, t2, key_limit=lim)
    assert np.array_equal(x2[:, :P + 2 * b], x[:, :P + 2 * b])
    assert np.abs(x2[0, P + 2 * b] - x[0, P + 2 * b]).max() > 1e-6
    assert np.abs(x2[0, P + 3 * b] - x[0, P + 3 * b]).max() > 1e-6
    t0 = draft_[:, :24]
    np.testing.assert_allclose(forward(W, t0, key_limit=block_key_limit(0, 24, 32)), forward(W, t0),
                               rtol=0, atol=0)


def test_draft_select_by_hand():
    m = np.array([[True, True, True, True, False, True]])
    c = np.array([[0.10, 0.70, 0.30, 0.70, 0.99, 0.20]])
    # 5 masked, 5 steps left: quota 1; nothing >= 0.8 -> the most confident
    # masked slot; 0.70 twice -> the lower position (1)
    assert draft_select(m, c, 0.8, 5)[0].tolist() == [False, True, False, False, False, False]
    # quota ceil(5/2) = 3: slots 1, 3 (0.70) then 2 (0.30)
    assert draft_select(m, c, 0.8, 2)[0].tolist() == [False, True, True, True, False, False]
    # threshold 0.25 admits 3 masked slots (0.70, 0.30, 0.70) > quota 1
    assert draft_select(m, c, 0.25, 5)[0].tolist() == [False, True, True, True, False, False]
    # conf == threshold counts; the unmasked slot 4 is never taken
    assert draft_select(m, c, 0.30, 5)[0].tolist() == [False, True, True, True, False, False]
    # last step: everything still masked
    assert draft_select(m, c, 2.0, 1)[0].tolist() == [True, True, True, True, False, True]
    # no masked slot: nothing; rows are independent
    m2 = np.array([[False, False], [True, True]])
    c2 = np.array([[0.9, 0.9], [0.2, 0.4]])
    assert draft_select(m2, c2, 0.5, 2).tolist() == [[False, False], [False, True]]


def test_draft_loop(tiny):
    """Quota pacing without the threshold (every step unmasks ceil(n/r) slots
    and a block takes all its steps); a threshold <= 0 or one step per block
    fills a block in one pass with the top-1 of the all-[MASK] block; a block
    does not depend on the blocks after it."""
    w, W = tiny
    prompt, _, _ = make_inputs(w)
    P, b, steps = 16, 8, 4
    pr = prompt[:, :P]
    mid = w.model.mask_id
    out, st = draft(W, pr, 2 * b, b, steps, 2.0)
    assert st["block_steps"] == [steps, steps] and st["n_masked_left"] == 0
    # replay with per-step counts
    t = np.concatenate([pr, np.full((1, 2 * b), mid, dtype=pr.dtype)], 1)
    for k in range(2):
        for s in range(steps):
            t, info = draft_step(W, t, P, b, k, 2.0, steps - s)
            assert info["n_unmasked"] == b // steps
    assert np.array_equal(t[:, P:], out)
    # one pass per block: block 0 = top-1 of the forward of [prompt, all MASK] under the block mask
    one, st1 = draft(W, pr, 2 * b, b, 1, 2.0)
    zero, st0 = draft(W, pr, 2 * b, b, steps, 0.0)
    assert st1["block_steps"] == [1, 1] and st0["block_steps"] == [1, 1]
    assert np.array_equal(one, zero)
    t0 = np.concatenate([pr, np.full((1, b), mid, dtype=pr.dtype)], 1)
    x = forward(W, t0, key_limit=block_key_limit(P, P + b, b))
    assert np.array_equal(one[:, :b], lm_head_reduce(W, x[0, P:])["top1"][None, :])
    # causality: drafting 3 blocks starts with the 2-block draft
    three, _ = draft(W, pr, 3 * b, b, steps, 0.3)
    two, _ = draft(W, pr, 2 * b, b, steps, 0.3)
    assert np.array_equal(three[:, :2 * b], two)
    # ragged last block (5 positions): still filled
    rag, str_ = draft(W, pr, b + 5, b, steps, 0.3)
    assert np.array_equal(rag[:, :b], two[:, :b]) and str_["n_masked_left"] == 0
    assert max(str_["block_steps"]) <= steps


def test_draft_forward_block_is_prefix_forward(tiny):
    """The step's forward over [0, end of block k) gives the same block rows as
    a forward over the whole sequence under the block mask (later blocks
    invisible)."""
    w, W = tiny
    prompt, draft_, _ = make_inputs(w)
    P, b = 16, 8
    t = np.concatenate([prompt[:, :P], draft_[:, :3 * b]], 1)
    info = draft_forward_block(W, t, P, b, 1)
    x = forward(W, t, key_limit=block_key_limit(P, t.shape[1], b))
    red = lm_head_reduce(W, x[0, P + b:P + 2 * b])
    assert np.array_equal(info["top1"][0], red["top1"])
    np.testing.assert_allclose(info["conf"][0], red["conf"], rtol=1e-12)


def test_cascade_pass_accounting(tiny):
    """Sec. 4.2's cost K x T_d + T_r: with pure quota pacing every block uses
    its T_d steps; zero refinement passes return the draft; the refine stage
    is refine_ex on the finished draft; a refiner identical to the drafter
    still runs (flash-flash, Sec. 4.3)."""
    from oracle.draft import cascade
    from oracle.refine import refine_ex
    w, W = tiny
    prompt, _, _ = make_inputs(w)
    pr = prompt[:, :16]
    Ws = oracle.OracleWeights(w.model.replace(n_layers=1), 3)
    K, Td, b = 3, 4, 8
    r0, st0 = cascade(Ws, W, pr, K * b, b, Td, 2.0, 0, 0.5, 0.5)
    d, _ = draft(Ws, pr, K * b, b, Td, 2.0)
    assert np.array_equal(r0, d) and st0["passes"] == K * Td and st0["refine"]["steps_run"] == 0
    r, st = cascade(Ws, W, pr, K * b, b, Td, 2.0, 3, 0.2, 0.2)
    ref, rst = refine_ex(W, pr, d, None, 3, 0.2, 0.2)
    assert np.array_equal(r, ref) and st["passes"] == K * Td + rst["steps_run"]
    assert 1 <= rst["steps_run"] <= 3
    same, sst = cascade(W, W, pr, K * b, b, Td, 0.3, 2, 0.2, 0.2)
    assert sst["draft"]["steps_run"] <= K * Td and sst["passes"] == sst["draft"]["steps_run"] + \
        sst["refine"]["steps_run"]
