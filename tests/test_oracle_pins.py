"""Pins for the CPU oracle: known answers, closed forms, invariants and library
routines that fix each of its functions independently of the oracle itself."""

from __future__ import annotations

import math
import os

import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

import oracle
from oracle import weights as ow
from oracle.refine import (attention, edit_rule, lm_head_reduce, moe_ffn, refine, refine_step,
                           rms_norm, rope, route, softmax, swiglu, forward, layer_forward)
from tests.planted import PlantedWeights, zero_block
from workloads import MODELS, WORKLOADS, make_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- generator

def _kat_rows():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            w = [int(t, 16) for t in line.split()]
            rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


@pytest.mark.parametrize("ctr,key,expect", _kat_rows())
def test_philox_known_answers(ctr, key, expect):
    assert ow.philox4x32_10(ctr, key) == expect


def test_irwin_hall_matches_its_block_definition():
    # n for element i is the centred sum of the four 16-bit halves of the first
    # two output words of the block with counter (i_lo, i_hi, tid, 0).
    seed, tid = 0x1234_5678_9abc_def0, ow.tensor_id(3, ow.K_WO)
    idx = [0, 1, 77, 2 ** 32 + 5]
    n = ow.irwin_hall_at(seed, tid, np.array(idx, dtype=np.uint64))
    for i, ni in zip(idx, n):
        w = ow.philox4x32_10([i & 0xffffffff, i >> 32, tid, 0], [seed & 0xffffffff, seed >> 32])
        s = (w[0] & 0xffff) + (w[0] >> 16) + (w[1] & 0xffff) + (w[1] >> 16)
        assert ni == s - 131070
    # range form and indexed form agree
    a = ow.irwin_hall(seed, tid, 70, 10)
    b = ow.irwin_hall_at(seed, tid, np.arange(70, 80, dtype=np.uint64))
    assert np.array_equal(a, b)


def test_irwin_hall_distribution():
    # Sum of four independent uniforms on {0..65535}: mean 131070, variance
    # 4 * (65536^2 - 1) / 12.  The scaled sum follows the Irwin-Hall(4) law.
    N = 1 << 20
    n = ow.irwin_hall(7, ow.tensor_id(1, ow.K_WQ), 0, N).astype(np.float64)
    assert n.min() >= -131070 and n.max() <= 131070
    var = 4 * (65536.0 ** 2 - 1) / 12
    assert abs(n.mean()) < 5 * math.sqrt(var / N)
    assert abs(n.var() / var - 1) < 0.01
    u = (n + 131070) / 65535.0            # in [0, 4]

    def ih4_cdf(x):
        x = np.asarray(x, dtype=np.float64)
        out = np.zeros_like(x)
        for k in range(5):
            out += (-1) ** k * scipy.special.comb(4, k) * np.clip(x - k, 0, None) ** 4
        return out / math.factorial(4)

    ks = scipy.stats.kstest(u, ih4_cdf)
    assert ks.pvalue > 1e-4
    # different tensors / seeds give different streams
    m = ow.irwin_hall(7, ow.tensor_id(1, ow.K_WK), 0, 1024)
    m2 = ow.irwin_hall(8, ow.tensor_id(1, ow.K_WQ), 0, 1024)
    assert not np.array_equal(n[:1024].astype(np.int32), m)
    assert not np.array_equal(n[:1024].astype(np.int32), m2)


def test_weight_values_are_bf16_and_scaled():
    c = ow.scale_constant(0.02)
    n = ow.irwin_hall(0, ow.tensor_id(2, ow.K_WV), 0, 1 << 18)
    v = ow.to_weight_values(n, c)
    bits = v.view(np.uint32)
    assert np.all(bits & 0xffff == 0)                      # on the bfloat16 grid
    exact = n.astype(np.float64) * float(c)
    nz = exact != 0
    rel = np.abs(v[nz] - exact[nz]) / np.abs(exact[nz])
    assert rel.max() <= 2.0 ** -8 * 1.0001                 # within half a bf16 ulp
    assert abs(v.std() / 0.02 - 1) < 0.01
    # RNE ties: a float32 exactly halfway between two bf16 values rounds to even
    t = torch.tensor([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8], dtype=torch.float32)
    assert t.to(torch.bfloat16).to(torch.float32).tolist() == [1.0, 1.0 + 2 ** -6]


# ---------------------------------------------------------------- primitives

def test_rms_norm_closed_forms():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 64))
    g = rng.standard_normal(64)
    # constant row c*1: output = g * c / sqrt(c^2 + eps)
    c, eps = -3.0, 1e-6
    y = rms_norm(np.full((1, 64), c), np.ones(64), eps)
    assert np.allclose(y, c / math.sqrt(c * c + eps), rtol=1e-15)
    # positive scale invariance (eps = 0) and unit mean square
    assert np.allclose(rms_norm(7.5 * x, g, 0.0), rms_norm(x, g, 0.0), rtol=1e-13)
    assert np.allclose(np.mean(rms_norm(x, np.ones(64), 0.0) ** 2, axis=-1), 1.0, rtol=1e-13)


def test_rope_pins():
    rng = np.random.default_rng(1)
    S, n, hd = 9, 3, 16
    x = rng.standard_normal((S, n, hd))
    pos = np.arange(S)
    y = rope(x, pos, 10000.0)
    # position 0 is the identity; norms are preserved
    assert np.allclose(y[0], x[0], rtol=0, atol=0)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    # complex form: (x_i + i x_{i+hd/2}) * exp(i * pos * theta^(-2i/hd))
    half = hd // 2
    z = x[..., :half] + 1j * x[..., half:]
    inv = 10000.0 ** (-np.arange(half) * 2.0 / hd)
    zr = z * np.exp(1j * pos[:, None, None] * inv[None, None, :])
    assert np.allclose(y[..., :half], zr.real, atol=1e-13)
    assert np.allclose(y[..., half:], zr.imag, atol=1e-13)
    # single pair with unit frequency: [1, 0] at position p -> [cos p, sin p]
    one = rope(np.tile(np.array([1.0, 0.0]), (S, 1, 1)), pos, 10000.0)
    assert np.allclose(one[:, 0, 0], np.cos(pos)) and np.allclose(one[:, 0, 1], np.sin(pos))
    # scores depend only on the position offset
    q = rng.standard_normal((1, 1, hd))
    k = rng.standard_normal((1, 1, hd))
    def score(pq, pk):
        a = rope(q, np.array([pq]), 10000.0)
        b = rope(k, np.array([pk]), 10000.0)
        return float(np.sum(a * b))
    assert math.isclose(score(3, 1), score(10, 8), rel_tol=1e-12)
    assert math.isclose(score(0, 5), score(100, 105), rel_tol=1e-12)


def test_softmax_matches_scipy():
    z = np.random.default_rng(2).standard_normal((4, 33)) * 10
    assert np.allclose(softmax(z), scipy.special.softmax(z, axis=-1), rtol=1e-14)


def test_attention_length_one_returns_v():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 8, 16))
    k = rng.standard_normal((1, 2, 16))
    v = rng.standard_normal((1, 2, 16))
    o = attention(q, k, v)
    assert np.allclose(o, np.repeat(v, 4, axis=1), rtol=1e-15)


def test_attention_zero_query_is_mean_over_all_keys():
    # A causal mask would give prefix means instead.
    rng = np.random.default_rng(4)
    S = 13
    q = np.zeros((S, 4, 8))
    k = rng.standard_normal((S, 4, 8))
    v = rng.standard_normal((S, 4, 8))
    o = attention(q, k, v)
    assert np.allclose(o, np.broadcast_to(v.mean(axis=0), o.shape), rtol=1e-13)


def test_attention_matches_torch_sdpa_noncausal_gqa():
    rng = np.random.default_rng(5)
    S, H, KV, hd = 37, 8, 2, 32
    q = rng.standard_normal((S, H, hd))
    k = rng.standard_normal((S, KV, hd))
    v = rng.standard_normal((S, KV, hd))
    o = attention(q, k, v)
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(np.repeat(k, H // KV, axis=1)).permute(1, 0, 2)
    tv = torch.from_numpy(np.repeat(v, H // KV, axis=1)).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=False)
    assert np.allclose(o, ref.permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-13)


def test_attention_permutation_equivariance():
    rng = np.random.default_rng(6)
    S = 11
    q, k, v = (rng.standard_normal((S, 2, 8)) for _ in range(3))
    perm = rng.permutation(S)
    o = attention(q, k, v)
    op = attention(q[perm], k[perm], v[perm])
    assert np.allclose(op, o[perm], rtol=1e-13)


def test_swiglu_pins():
    rng = np.random.default_rng(7)
    h = rng.standard_normal((5, 16))
    wg, wu = rng.standard_normal((24, 16)), rng.standard_normal((24, 16))
    wd = rng.standard_normal((16, 24))
    g, u = h @ wg.T, h @ wu.T
    ref = (g * scipy.special.expit(g) * u) @ wd.T
    assert np.allclose(swiglu(h, wg, wu, wd), ref, rtol=1e-12)
    assert np.all(swiglu(h, wg, wu, np.zeros_like(wd)) == 0)


def _moe_layer(rng, E, F, d, n_shared):
    r = lambda *s: rng.standard_normal(s) * 0.3
    return {"w_router": r(E, d),
            "experts": [(r(F, d), r(F, d), r(d, F)) for _ in range(E)],
            "shared": [(r(F, d), r(F, d), r(d, F)) for _ in range(n_shared)]}


def test_route_ties_go_to_lower_id_and_weights_renormalise():
    h = np.ones((1, 4))
    wr = np.array([[1.0, 0, 0, 0], [2.0, 0, 0, 0], [2.0, 0, 0, 0], [2.0, 0, 0, 0], [0.5, 0, 0, 0]])
    ids, w, gap = route(h, wr, 2)
    assert ids.tolist() == [[1, 2]]
    assert np.allclose(w, 0.5) and gap[0] == 0.0
    rng = np.random.default_rng(8)
    hh = rng.standard_normal((20, 8))
    wr2 = rng.standard_normal((6, 8))
    ids, w, _ = route(hh, wr2, 6, decide_bf16=False)   # k = E: full softmax mixture
    p = scipy.special.softmax(hh @ wr2.T, axis=-1)
    assert np.allclose(np.take_along_axis(p, ids, -1), w, rtol=1e-13)
    _, w3, _ = route(hh, wr2, 3, decide_bf16=False)
    assert np.allclose(w3.sum(-1), 1.0, rtol=1e-14)


def test_moe_expert_permutation_invariance():
    rng = np.random.default_rng(9)
    E, F, d = 6, 12, 10
    L = _moe_layer(rng, E, F, d, 1)
    h = rng.standard_normal((30, d))
    out, _, _, _ = moe_ffn(h, L, 2)
    perm = rng.permutation(E)
    Lp = {"w_router": L["w_router"][perm], "experts": [L["experts"][i] for i in perm],
          "shared": L["shared"]}
    outp, _, _, _ = moe_ffn(h, Lp, 2)
    assert np.allclose(out, outp, rtol=1e-12, atol=1e-14)


def test_moe_reductions():
    rng = np.random.default_rng(10)
    d, F = 10, 12
    h = rng.standard_normal((25, d))
    one = _moe_layer(rng, 1, F, d, 0)                      # E = 1, k = 1: dense SwiGLU
    out, _, _, _ = moe_ffn(h, one, 1)
    assert np.allclose(out, swiglu(h, *one["experts"][0]), rtol=1e-13)
    same = _moe_layer(rng, 5, F, d, 0)                     # identical experts: weights sum to 1
    same["experts"] = [same["experts"][0]] * 5
    out, _, _, _ = moe_ffn(h, same, 3)
    assert np.allclose(out, swiglu(h, *same["experts"][0]), rtol=1e-12)
    sh = _moe_layer(rng, 4, F, d, 1)                       # shared expert is always added
    routed = dict(sh, shared=[])
    a, _, _, _ = moe_ffn(h, sh, 2)
    b, _, _, _ = moe_ffn(h, routed, 2)
    assert np.allclose(a - b, swiglu(h, *sh["shared"][0]), rtol=1e-12, atol=1e-13)


def test_decisions_read_bf16_rounded_operands():
    from oracle.refine import bf16_round
    # representable values are unchanged; ties go to even; float64 is rounded to
    # float32 first (as the kernels round their fp32 activations), so
    # 1 + 2^-8 + 2^-30 -> 1 + 2^-8 (fp32) -> 1.0 (bf16 tie to even).
    assert np.array_equal(bf16_round(np.array([1.0, -0.5, 3.0, 2.0 ** -20])), [1.0, -0.5, 3.0, 2.0 ** -20])
    assert bf16_round(np.array([1.0 + 2 ** -8]))[0] == 1.0
    assert bf16_round(np.array([1.0 + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6
    assert bf16_round(np.array([1.0 + 2 ** -8 + 2 ** -30]))[0] == 1.0
    # inputs already on the bf16 grid: both decision precisions agree exactly
    rng = np.random.default_rng(21)
    h = bf16_round(rng.standard_normal((40, 16)))
    wr = rng.standard_normal((8, 16))
    a = route(h, wr, 3, decide_bf16=True)
    b = route(h, wr, 3, decide_bf16=False)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    # the router ranks on the rounded input: a near tie that rounding reverses
    wr2 = np.array([[1.0, 0.0], [0.0, 1.0]])
    hh = np.array([[1.0 + 2 ** -9, 1.0 + 2 ** -10]])      # exact: expert 0 ahead; bf16: tie -> lower id 0
    assert route(hh, wr2, 1, decide_bf16=False)[0][0, 0] == 0
    assert route(hh, wr2, 1, decide_bf16=True)[0][0, 0] == 0
    hh = np.array([[1.0 + 2 ** -10, 1.0 + 2 ** -9]])      # exact: expert 1 ahead; bf16: tie -> 0
    assert route(hh, wr2, 1, decide_bf16=False)[0][0, 0] == 1
    assert route(hh, wr2, 1, decide_bf16=True)[0][0, 0] == 0


# ---------------------------------------------------------------- reduction

class _HeadOnly:
    def __init__(self, shape, wlm):
        self.shape = shape
        self._w = wlm

    def lm_head(self):
        return self._w

    def final_norm(self):
        return np.ones(self.shape.d_model)


def test_lm_head_reduce_against_explicit_softmax():
    rng = np.random.default_rng(11)
    shape = MODELS["tiny"].replace(vocab=300, d_model=32)
    wlm = rng.standard_normal((300, 32)) * 0.5
    x = rng.standard_normal((17, 32))
    red = lm_head_reduce(_HeadOnly(shape, wlm), x, row_chunk=5, want_logits=True, decide_bf16=False)
    z = (x / np.sqrt(np.mean(x * x, -1, keepdims=True) + shape.norm_eps)) @ wlm.T
    p = scipy.special.softmax(z, axis=-1)
    assert np.array_equal(red["top1"], np.argmax(z, -1))
    assert np.allclose(red["conf"], p.max(-1), rtol=1e-12)
    srt = np.sort(z, -1)
    assert np.allclose(red["margin"], srt[:, -1] - srt[:, -2], rtol=1e-12)
    assert np.allclose(red["max_logit"], srt[:, -1], rtol=1e-13)


def test_lm_head_reduce_degenerate_cases():
    shape = MODELS["tiny"].replace(vocab=64, d_model=16)
    x = np.random.default_rng(12).standard_normal((3, 16))
    red = lm_head_reduce(_HeadOnly(shape, np.zeros((64, 16))), x)
    assert np.all(red["top1"] == 0) and np.allclose(red["conf"], 1 / 64, rtol=1e-15)
    w = np.zeros((64, 16))
    w[41] = 50.0                                             # planted winner
    red = lm_head_reduce(_HeadOnly(shape, w), np.abs(x) + 0.1)
    assert np.all(red["top1"] == 41) and np.all(red["conf"] > 0.999999)


# ---------------------------------------------------------------- editing rule

def test_edit_rule_cases():
    mask_id = 9
    draft = np.array([[1, 9, 3, 9, 5]])
    top1 = np.array([[1, 4, 7, 9, 6]])
    conf = np.array([[0.95, 0.5, 0.7, 0.99, 0.2]])
    new, unm, ed = edit_rule(draft, top1, conf, 0.6, mask_id)
    assert new.tolist() == [[1, 9, 7, 9, 5]] and (unm, ed) == (0, 1)
    new, unm, ed = edit_rule(draft, top1, conf, 0.0, mask_id)  # tau <= 0: take every top-1 but [MASK]
    assert new.tolist() == [[1, 4, 7, 9, 6]] and (unm, ed) == (1, 2)
    new, unm, ed = edit_rule(draft, top1, conf, 1.5, mask_id)  # tau > 1: nothing moves
    assert new.tolist() == draft.tolist() and (unm, ed) == (0, 0)
    new, _, _ = edit_rule(draft, top1, conf, 0.5, mask_id)      # conf == tau takes (>=)
    assert new[0, 1] == 4


def test_edit_rule_ex_cases():
    """Two thresholds and the EOS count, worked by hand from the rule."""
    from oracle.refine import edit_rule_ex
    mask_id, eos = 9, 7
    draft = np.array([[9, 3, 9, 4, 5]])
    top1 = np.array([[2, 3, 9, 6, 7]])
    conf = np.array([[0.5, 0.99, 0.99, 0.7, 0.95]])
    # [MASK]->2 (0.5 >= 0.4); 3 unchanged (same token); [MASK] top-1 is [MASK]:
    # stays; 4->6 refused (0.7 < 0.9); 5->7 (0.95 >= 0.9) writes the EOS id
    new, unm, ed, ne = edit_rule_ex(draft, top1, conf, 0.4, 0.9, mask_id, eos)
    assert new.tolist() == [[2, 3, 9, 4, 7]] and (unm, ed, ne) == (1, 1, 1)
    # swapped thresholds: the unmask is refused (0.5 < 0.9), both edits pass
    new, unm, ed, ne = edit_rule_ex(draft, top1, conf, 0.9, 0.4, mask_id, eos)
    assert new.tolist() == [[9, 3, 9, 6, 7]] and (unm, ed, ne) == (0, 2, 1)
    # eos disabled: no count; a slot already holding the EOS id is not "produced"
    assert edit_rule_ex(draft, top1, conf, 0.4, 0.9, mask_id, -1)[3] == 0
    d2 = np.array([[9, 3, 9, 4, 7]])
    assert edit_rule_ex(d2, top1, conf, 0.4, 0.9, mask_id, eos)[3] == 0
    # edit threshold > 1: only [MASK] slots move; unmask threshold > 1: only real tokens
    rng = np.random.default_rng(3)
    dr = rng.integers(0, 12, size=(4, 50))
    t1 = rng.integers(0, 12, size=(4, 50))
    cf = rng.random((4, 50))
    n1 = edit_rule_ex(dr, t1, cf, 0.3, 1.5, 11)[0]
    assert np.all((n1 == dr) | (dr == 11))
    n2 = edit_rule_ex(dr, t1, cf, 1.5, 0.3, 11)[0]
    assert np.all((n2 == dr) | (dr != 11))
    # equal thresholds reduce to the single-threshold rule
    for tau in (0.0, 0.3, 0.7, 1.1):
        a = edit_rule_ex(dr, t1, cf, tau, tau, 11, -1)
        b = edit_rule(dr, t1, cf, tau, 11)
        assert np.array_equal(a[0], b[0]) and a[1:3] == b[1:3]


# ---------------------------------------------------------------- composed step

def test_identity_blocks_closed_form():
    # One-hot embeddings, identity LM head, blocks that are the identity on the
    # residual stream: top1 = the token itself and conf = e^sqrt(d) / (e^sqrt(d) + V - 1).
    shape = MODELS["tiny"].replace(vocab=32, d_model=64, n_heads=2, n_kv_heads=2, head_dim=32,
                                   ffn_dim=48, n_layers=2)
    E = np.eye(32, 64)
    W = PlantedWeights(shape, E, np.eye(32, 64), [zero_block(shape), zero_block(shape)])
    tokens = np.array([[3, 7, 1, 30, 5, 5, 0]])
    x = forward(W, tokens)
    assert np.array_equal(x, E[tokens])
    red = lm_head_reduce(W, x[0], decide_bf16=False)
    a = math.exp(math.sqrt(64 / (1 + 64 * shape.norm_eps)))
    assert np.array_equal(red["top1"], tokens[0])
    assert np.allclose(red["conf"], a / (a + 31), rtol=1e-12)


def test_identity_blocks_closed_form_moe():
    shape = MODELS["small_moe"].replace(vocab=40, d_model=64, n_heads=4, n_kv_heads=2,
                                        head_dim=16, n_experts=4, top_k=2, expert_ffn_dim=8,
                                        n_layers=1)
    E = np.eye(40, 64)
    W = PlantedWeights(shape, E, np.eye(40, 64), [zero_block(shape)])
    tokens = np.array([[4, 9, 39, 2]])
    x = forward(W, tokens)
    assert np.array_equal(x, E[tokens])


@pytest.fixture(scope="module")
def tiny():
    w = WORKLOADS["tiny"]
    return w, oracle.OracleWeights(w.model, w.weight_seed)


def test_forward_is_bidirectional(tiny):
    # Changing the last token changes the residual stream at the first position.
    w, W = tiny
    prompt, draft, _ = make_inputs(w)
    t = np.concatenate([prompt, draft], 1)
    t2 = t.copy()
    t2[0, -1] = (t2[0, -1] + 1) % (w.model.vocab - 1)
    a, b = forward(W, t), forward(W, t2)
    assert np.abs(a[0, 0] - b[0, 0]).max() > 1e-6


def test_refine_invariants(tiny):
    w, W = tiny
    prompt, draft, mask = make_inputs(w)
    mid = w.model.mask_id
    # empty mask set and tau > 1: tokens unchanged, one pass, loop stops
    out, st = refine(W, prompt, draft, None, 4, 1.01)
    assert np.array_equal(out, draft) and st["steps_run"] == 1
    # n_steps = 0: only the mask set is applied
    out, st = refine(W, prompt, draft, mask, 0, 0.5)
    assert st["steps_run"] == 0 and np.array_equal(out == mid, mask)
    # tau <= 0: every draft slot takes its top-1 (never [MASK]); prompt fixed
    t = np.concatenate([prompt, np.where(mask, mid, draft)], 1).astype(np.int32)
    t1, info = refine_step(W, t, w.prompt_len, 0.0)
    assert np.array_equal(t1[:, :w.prompt_len], prompt)
    assert np.array_equal(t1[:, w.prompt_len:], info["top1"])
    assert info["n_unmasked"] == int(mask.sum())
    # the edited set shrinks as tau grows (same input)
    taus = np.quantile(info["conf"], [0.2, 0.5, 0.8])
    moved = [refine_step(W, t, w.prompt_len, tau)[0] != t for tau in taus]
    assert np.all(moved[1] <= moved[0]) and np.all(moved[2] <= moved[1])
    # refine(a) then refine(b) == refine(a + b); masks never increase
    tau = float(np.quantile(info["conf"], 0.6))
    a, sa = refine(W, prompt, draft, mask, 1, tau)
    ab, sab = refine(W, prompt, a, None, 2, tau)
    full, sf = refine(W, prompt, draft, mask, 3, tau)
    assert np.array_equal(ab, full)
    assert (ab == mid).sum() <= (a == mid).sum() <= mask.sum()


def test_refine_ex_loop(tiny):
    """Equal thresholds without EOS: the same run as refine (and stop_reason 1
    or 0); with an EOS id that the first pass writes, the loop ends after that
    pass (stop_reason 2) where the same run without EOS goes on."""
    from oracle.refine import refine_ex
    w, W = tiny
    prompt, draft, mask = make_inputs(w)
    P = w.prompt_len
    t = np.concatenate([prompt, np.where(mask, w.model.mask_id, draft)], 1).astype(np.int32)
    _, info = refine_step(W, t, P, 0.0)
    tau = float(np.quantile(info["conf"], 0.5))
    a, sa = refine(W, prompt, draft, mask, 3, tau)
    b, sb = refine_ex(W, prompt, draft, mask, 3, tau, tau)
    assert np.array_equal(a, b) and sa["steps_run"] == sb["steps_run"]
    assert sb["stop_reason"] == (1 if sb["per_step"][-1]["n_unmasked"] + sb["per_step"][-1]["n_edited"] == 0 else 0)
    # tau <= 0 makes pass 1 write every top-1: take one written token as EOS
    t1, inf1 = refine_step(W, t, P, 0.0)
    written = t1[:, P:][t1[:, P:] != t[:, P:]]
    eos = int(written[0])
    c, sc = refine_ex(W, prompt, draft, mask, 3, 0.0, 0.0, eos)
    assert sc["steps_run"] == 1 and sc["stop_reason"] == 2 and np.array_equal(c, t1[:, P:])
    d, sd = refine_ex(W, prompt, draft, mask, 3, 0.0, 0.0, -1)
    assert sd["steps_run"] > 1 or sd["stop_reason"] == 1


def test_rope_positions_in_forward(tiny):
    """Shifting every position by the same amount leaves the forward unchanged
    (RoPE scores depend on offsets only); shifting only the draft positions
    changes it (the positions reach the blocks)."""
    w, W = tiny
    prompt, draft, _ = make_inputs(w)
    t = np.concatenate([prompt, draft], 1)
    S = t.shape[1]
    base = forward(W, t)
    np.testing.assert_allclose(forward(W, t, positions=np.arange(S) + 37), base, rtol=0, atol=1e-9)
    shifted = np.concatenate([np.arange(w.prompt_len), w.prompt_len + 16 + np.arange(S - w.prompt_len)])
    assert np.abs(forward(W, t, positions=shifted) - base).max() > 1e-6


def test_refine_local_schedules(tiny):
    """One stage spanning the draft is refine_ex; with an empty prompt each
    chunk equals refine_ex of the chunk alone (positions enter through offsets
    only); a chunk's result does not depend on the other chunks."""
    from oracle.refine import refine_ex, refine_local
    w, W = tiny
    prompt, draft, mask = make_inputs(w)
    P, D = w.prompt_len, w.draft_len
    t = np.concatenate([prompt, np.where(mask, w.model.mask_id, draft)], 1).astype(np.int32)
    _, info = refine_step(W, t, P, 0.0)
    tau = float(np.quantile(info["conf"], 0.5))
    a, sa = refine_local(W, prompt, draft, mask, [(D, 3)], tau, tau)
    b, sb = refine_ex(W, prompt, draft, mask, 3, tau, tau)
    assert np.array_equal(a, b) and sa["steps_run"] == sb["steps_run"] and sa["stop_reason"] == sb["stop_reason"]
    # empty prompt, two chunks of 32: chunk c alone at positions 0..31
    empty = np.zeros((1, 0), dtype=prompt.dtype)
    c, sc = refine_local(W, empty, draft, mask, [(32, 2)], 0.0, 0.0)
    for c0 in (0, 32):
        alone, _ = refine_ex(W, empty, draft[:, c0:c0 + 32], mask[:, c0:c0 + 32], 2, 0.0, 0.0)
        assert np.array_equal(c[:, c0:c0 + 32], alone)
    # chunk independence: changing the second chunk leaves the first one's result
    d2 = draft.copy()
    d2[:, 40:] = (d2[:, 40:] + 1) % (w.model.vocab - 1)
    e, _ = refine_local(W, prompt, d2, mask, [(32, 2)], 0.0, 0.0)
    f, _ = refine_local(W, prompt, draft, mask, [(32, 2)], 0.0, 0.0)
    assert np.array_equal(e[:, :32], f[:, :32]) and not np.array_equal(e[:, 32:], f[:, 32:])


def test_layer_forward_collect_consistent(tiny):
    w, W = tiny
    prompt, draft, _ = make_inputs(w)
    t = np.concatenate([prompt, draft], 1)
    x, infos, inputs = forward(W, t, collect=True)
    y = inputs[-1]
    y, _ = layer_forward(w.model, W.layer(w.model.n_layers - 1), y)
    assert np.array_equal(x, y)


def test_block_wiring_uniform_attention_closed_form():
    # Wq = 0 makes every attention row uniform, Wv = Wo = I and a zero FFN, so
    # each position gains the mean over all positions of rms_norm(x).
    shape = MODELS["tiny"].replace(vocab=16, d_model=32, n_heads=2, n_kv_heads=2, head_dim=16,
                                   ffn_dim=8, n_layers=1)
    L = zero_block(shape)
    L["wq"] = np.zeros_like(L["wq"])
    L["wv"] = np.eye(32)
    L["wo"] = np.eye(32)
    x = np.random.default_rng(13).standard_normal((2, 5, 32))
    y, _ = layer_forward(shape, L, x)
    h = x / np.sqrt(np.mean(x * x, -1, keepdims=True) + shape.norm_eps)
    assert np.allclose(y, x + h.mean(axis=1, keepdims=True), rtol=1e-12, atol=1e-13)


def test_block_wiring_ffn_closed_form():
    # Zero attention output; gate = up = down = I: each position gains
    # silu(h) * h with h = rms_norm(x).
    shape = MODELS["tiny"].replace(vocab=16, d_model=32, n_heads=2, n_kv_heads=2, head_dim=16,
                                   ffn_dim=32, n_layers=1)
    L = zero_block(shape)
    L["w_gate"] = np.eye(32)
    L["w_up"] = np.eye(32)
    L["w_down"] = np.eye(32)
    x = np.random.default_rng(14).standard_normal((1, 6, 32))
    y, _ = layer_forward(shape, L, x)
    h = x / np.sqrt(np.mean(x * x, -1, keepdims=True) + shape.norm_eps)
    assert np.allclose(y, x + h * scipy.special.expit(h) * h, rtol=1e-12, atol=1e-13)


def test_layer_forward_rows_matches_the_full_block():
    """The row-subset block (used to check large batches on sampled tokens)
    equals the full block at those positions, dense and MoE."""
    from oracle.refine import layer_forward_rows
    for shape in (MODELS["tiny"].replace(n_layers=1),
                  MODELS["small_moe"].replace(vocab=96, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16,
                                              n_experts=6, top_k=2, expert_ffn_dim=16, n_layers=1)):
        W = oracle.OracleWeights(shape, 5)
        rng = np.random.default_rng(2)
        x = rng.standard_normal((2, 19, shape.d_model))
        full, info = layer_forward(shape, W.layer(0), x)
        rows = np.array([0, 3, 4, 18])
        part, pinfo = layer_forward_rows(shape, W.layer(0), x[1], rows)
        assert np.allclose(part, full[1, rows], rtol=1e-12, atol=1e-12)
        if shape.n_experts:
            assert np.array_equal(pinfo["route_ids"], info["route_ids"][1, rows])
