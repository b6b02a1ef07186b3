"""Plain float64 CPU implementation of one refinement step and of the refine loop.

CPU oracle -- test infrastructure only.  Only tests/, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with the
GPU library and imports nothing from it.

What is computed (paper: Sec. 4.2 "Bidirectional Refinement"; App. C.4 and
Table 10 for the threshold and the early stop):

  * The refiner receives the prompt x and a complete draft y.  Prompt tokens
    stay fixed; every draft position may be revised using the whole sequence
    (Sec. 4.2).  One refinement pass is one full-sequence bidirectional
    forward: attention has no causal or block mask of any kind.
  * Each draft position's logits are reduced to the top-1 token and its
    confidence, the softmax probability of that token over the full vocabulary.
  * Editing rule (the paper names a threshold editing rule with one refine
    threshold, Table 10, but does not spell it out; the reading used here):
    all draft positions are decided from the same forward pass; a position
    whose top-1 is not [MASK] and whose confidence is >= tau takes the top-1
    token.  A [MASK] slot that changes counts as unmasked, a real token that
    changes counts as edited.  Prompt slots are never written.
  * The pass budget is an upper bound: the loop stops after a pass in which no
    position changed, since the next pass would see identical input (App. C.4).

The refiner's architecture is not described in the paper (Sec. 5.1); this
oracle uses a pre-norm RMSNorm transformer with rotate-half RoPE,
softmax-routed top-k SwiGLU experts (renormalised over the selected k) plus an
always-on shared expert, and an untied LM head.

All arithmetic is float64 on weights that hold bfloat16 values; there is no
blocking, fusion or reordering beyond the matrix products themselves.

Integer decisions taken from floating-point values -- which experts a token is
routed to, and the top-1 token of each draft position -- are taken from the
exact float64 logits.  A bf16-rounded GPU path can decide differently only
where those logits nearly tie; the parity tests exempt such positions by the
tolerances of the method's contract (top-1/top-2 margin and distance from the
threshold, router top-k gap) and check each exemption against the measured
logit error.  decide_bf16=True is a diagnostic only: the router and the LM
head then read their input activations rounded to bfloat16 first (the GEMM
operand precision of the kernels), which shows how many exempt decisions the
operand rounding alone explains.
"""

from __future__ import annotations

import numpy as np
import torch

F64 = np.float64


def bf16_round(x: np.ndarray) -> np.ndarray:
    """x rounded float64 -> float32 -> bfloat16 (round to nearest even, torch), as float64."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float64).numpy()


# ---------------------------------------------------------------- primitives

def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = x.astype(F64, copy=False)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g.astype(F64)


def rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding.  x: [S, n_heads, hd]; positions: [S].

    Pair (i, i + hd/2) is rotated by angle pos * theta**(-2i/hd).
    """
    hd = x.shape[-1]
    half = hd // 2
    inv_freq = theta ** (-(np.arange(half, dtype=F64) * 2.0) / hd)
    ang = positions.astype(F64)[:, None] * inv_freq[None, :]          # [S, half]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def softmax(z: np.ndarray, axis: int = -1) -> np.ndarray:
    m = np.max(z, axis=axis, keepdims=True)
    e = np.exp(z - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, key_limit: np.ndarray | None = None) -> np.ndarray:
    """Non-causal attention: every query attends to all S keys.

    q: [S, H, hd]; k, v: [S, KV, hd] with H a multiple of KV (query head h reads
    key/value head h // (H // KV)).  Returns [S, H, hd].  With key_limit [S],
    query i attends to keys 0 .. key_limit[i]-1 only (the block-causal mask of
    block-AR drafting, Sec. 3.3); the refiner passes none.
    """
    S, H, hd = q.shape
    KV = k.shape[1]
    group = H // KV
    out = np.empty((S, H, hd), dtype=F64)
    scale = 1.0 / np.sqrt(hd)
    allowed = None
    if key_limit is not None:
        allowed = np.arange(k.shape[0])[None, :] < np.asarray(key_limit)[:, None]
    for h in range(H):
        kv = h // group
        scores = (q[:, h, :] @ k[:, kv, :].T) * scale                 # [S, S]
        if allowed is not None:
            scores = np.where(allowed, scores, -np.inf)
        out[:, h, :] = softmax(scores, axis=-1) @ v[:, kv, :]
    return out


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def swiglu(h: np.ndarray, w_gate, w_up, w_down) -> np.ndarray:
    """(silu(h Wg^T) * (h Wu^T)) Wd^T with W stored [out, in]."""
    g = h @ w_gate.astype(F64).T
    u = h @ w_up.astype(F64).T
    return (silu(g) * u) @ w_down.astype(F64).T


def route(h: np.ndarray, w_router, k: int, decide_bf16: bool = False, return_logits: bool = False):
    """Softmax router, top-k (ties go to the lower expert id), renormalised.

    Returns ids [T, k], weights [T, k] and the logit gap between the k-th and
    (k+1)-th ranked experts (inf when k == E), and with return_logits also the
    router logits z [T, E].  With decide_bf16 (a diagnostic) the router reads h
    rounded to bfloat16.
    """
    if decide_bf16:
        h = bf16_round(h)
    z = h @ w_router.astype(F64).T                                     # [T, E]
    p = softmax(z, axis=-1)
    order = np.argsort(-z, axis=-1, kind="stable")                     # desc, ties -> lower id
    ids = order[:, :k]
    sel = np.take_along_axis(p, ids, axis=-1)
    w = sel / np.sum(sel, axis=-1, keepdims=True)
    E = z.shape[-1]
    if k < E:
        zs = np.take_along_axis(z, order[:, k - 1:k + 1], axis=-1)
        gap = zs[:, 0] - zs[:, 1]
    else:
        gap = np.full(z.shape[0], np.inf)
    if return_logits:
        return ids, w, gap, z
    return ids, w, gap


def moe_ffn(h: np.ndarray, L: dict, k: int, decide_bf16: bool = False):
    """Sum over the selected experts of w_j * SwiGLU_j(h), plus the shared experts."""
    T = h.shape[0]
    ids, w, gap, z = route(h, L["w_router"], k, decide_bf16, return_logits=True)
    out = np.zeros_like(h)
    for e in range(len(L["experts"])):
        rows, slot = np.nonzero(ids == e)
        if rows.size == 0:
            continue                      # an expert's weights are only read if a token uses it
        wg, wu, wd = L["experts"][e]
        y = swiglu(h[rows], wg, wu, wd)
        out[rows] += w[rows, slot][:, None] * y
    for (wg, wu, wd) in L["shared"]:
        out += swiglu(h, wg, wu, wd)
    return out, ids, gap, z


# ---------------------------------------------------------------- forward

def layer_forward(shape, L: dict, x: np.ndarray, decide_bf16: bool = False, positions: np.ndarray | None = None,
                  key_limit: np.ndarray | None = None):
    """One pre-norm block over x [B, S, d] (all positions; no attention mask
    unless key_limit [S] is given, see attention); positions [S] (default
    0..S-1) are the RoPE positions of the S tokens."""
    B, S, d = x.shape
    H, KV, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
    pos = np.arange(S) if positions is None else np.asarray(positions)
    x = x.astype(F64, copy=True)
    info = {"route_gap": None, "route_ids": None, "router_logits": None}
    attn = np.empty((B, S, H * hd), dtype=F64)
    for b in range(B):
        h = rms_norm(x[b], L["g1"], shape.norm_eps)
        q = (h @ L["wq"].astype(F64).T).reshape(S, H, hd)
        kk = (h @ L["wk"].astype(F64).T).reshape(S, KV, hd)
        v = (h @ L["wv"].astype(F64).T).reshape(S, KV, hd)
        q = rope(q, pos, shape.rope_theta)
        kk = rope(kk, pos, shape.rope_theta)
        attn[b] = attention(q, kk, v, key_limit).reshape(S, H * hd)
    x += attn @ L["wo"].astype(F64).T
    h2 = rms_norm(x.reshape(B * S, d), L["g2"], shape.norm_eps)
    if shape.n_experts == 0:
        ffn = swiglu(h2, L["w_gate"], L["w_up"], L["w_down"])
    else:
        ffn, ids, gap, z = moe_ffn(h2, L, shape.top_k, decide_bf16)
        info["route_gap"] = gap.reshape(B, S)
        info["route_ids"] = ids.reshape(B, S, -1)
        info["router_logits"] = z.reshape(B, S, -1)
    x += ffn.reshape(B, S, d)
    return x, info


def layer_forward_rows(shape, L: dict, x_seq: np.ndarray, rows: np.ndarray, decide_bf16: bool = False):
    """The block of layer_forward for one sequence x_seq [S, d], evaluated only
    at the positions `rows`: keys and values come from all S positions, the
    queries and everything after attention (which is per position) from the
    selected ones.  Returns (x [len(rows), d], info for those rows)."""
    S, d = x_seq.shape
    H, KV, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
    rows = np.asarray(rows)
    x_seq = x_seq.astype(F64)
    h = rms_norm(x_seq, L["g1"], shape.norm_eps)
    q = (h[rows] @ L["wq"].astype(F64).T).reshape(len(rows), H, hd)
    kk = (h @ L["wk"].astype(F64).T).reshape(S, KV, hd)
    v = (h @ L["wv"].astype(F64).T).reshape(S, KV, hd)
    q = rope(q, rows, shape.rope_theta)
    kk = rope(kk, np.arange(S), shape.rope_theta)
    x = x_seq[rows] + attention(q, kk, v).reshape(len(rows), H * hd) @ L["wo"].astype(F64).T
    h2 = rms_norm(x, L["g2"], shape.norm_eps)
    info = {"route_gap": None, "route_ids": None, "router_logits": None}
    if shape.n_experts == 0:
        x = x + swiglu(h2, L["w_gate"], L["w_up"], L["w_down"])
    else:
        ffn, ids, gap, z = moe_ffn(h2, L, shape.top_k, decide_bf16)
        x = x + ffn
        info["route_gap"], info["route_ids"], info["router_logits"] = gap, ids, z
    return x, info


def forward(W, tokens: np.ndarray, collect: bool = False, decide_bf16: bool = False,
            positions: np.ndarray | None = None, key_limit: np.ndarray | None = None):
    """Residual stream after the last layer (before the final norm): [B, S, d].

    With collect=True also returns per-layer infos and per-layer inputs;
    positions and key_limit as in layer_forward.
    """
    shape = W.shape
    x = W.embed_rows(np.asarray(tokens)).astype(F64)
    infos, inputs = [], []
    for l in range(shape.n_layers):
        if collect:
            inputs.append(x.copy())
        x, info = layer_forward(shape, W.layer(l), x, decide_bf16, positions, key_limit)
        infos.append(info)
    if collect:
        return x, infos, inputs
    return x


# ---------------------------------------------------------------- reduction

def lm_head_reduce(W, x_rows: np.ndarray, row_chunk: int = 256, want_logits: bool = False,
                   decide_bf16: bool = False):
    """Per row: logits z = (rms(x) g_f) Wlm^T over the full vocabulary (the
    normalised row rounded to bfloat16 when decide_bf16), then

      m     = max_v z_v
      top1  = min { v : z_v = m }           (first maximum)
      m2    = max_{v != top1} z_v           (runner-up logit)
      s     = sum_v exp(z_v - m)
      conf  = 1 / s                         (softmax probability of top1)
    """
    shape = W.shape
    wlm = W.lm_head().astype(F64)
    R = x_rows.shape[0]
    top1 = np.empty(R, dtype=np.int64)
    conf = np.empty(R, dtype=F64)
    m = np.empty(R, dtype=F64)
    m2 = np.empty(R, dtype=F64)
    logits = [] if want_logits else None
    for r0 in range(0, R, row_chunk):
        hx = rms_norm(x_rows[r0:r0 + row_chunk], W.final_norm(), shape.norm_eps)
        if decide_bf16:
            hx = bf16_round(hx)
        z = hx @ wlm.T
        t = np.argmax(z, axis=-1)
        mm = z[np.arange(z.shape[0]), t]
        zz = z.copy()
        zz[np.arange(z.shape[0]), t] = -np.inf
        s = np.sum(np.exp(z - mm[:, None]), axis=-1)
        top1[r0:r0 + row_chunk] = t
        m[r0:r0 + row_chunk] = mm
        m2[r0:r0 + row_chunk] = np.max(zz, axis=-1)
        conf[r0:r0 + row_chunk] = 1.0 / s
        if want_logits:
            logits.append(z)
    out = {"top1": top1, "conf": conf, "max_logit": m, "margin": m - m2}
    if want_logits:
        out["logits"] = np.concatenate(logits, axis=0)
    return out


# ---------------------------------------------------------------- editing rule

def edit_rule(draft: np.ndarray, top1: np.ndarray, conf: np.ndarray, tau: float, mask_id: int):
    """Simultaneous threshold update of all draft positions from one forward.

    draft, top1: [B, D] ints; conf: [B, D] floats.  A position takes its top-1
    token when top1 != mask_id and conf >= tau.
    """
    take = (top1 != mask_id) & (conf >= tau)
    new = np.where(take, top1, draft).astype(draft.dtype)
    changed = new != draft
    n_unmasked = int(np.sum(changed & (draft == mask_id)))
    n_edited = int(np.sum(changed & (draft != mask_id)))
    return new, n_unmasked, n_edited


def _reduce_draft(W, tokens: np.ndarray, prompt_len: int, decide_bf16: bool, positions: np.ndarray | None = None):
    """Forward over the whole sequence, then top-1 and confidence of every draft position."""
    B, S = tokens.shape
    D = S - prompt_len
    x = forward(W, tokens, decide_bf16=decide_bf16, positions=positions)
    red = lm_head_reduce(W, x[:, prompt_len:, :].reshape(B * D, -1), decide_bf16=decide_bf16)
    return {"top1": red["top1"].reshape(B, D), "conf": red["conf"].reshape(B, D),
            "max_logit": red["max_logit"].reshape(B, D), "margin": red["margin"].reshape(B, D)}


def refine_step(W, tokens: np.ndarray, prompt_len: int, tau: float, decide_bf16: bool = False):
    """One refinement pass over tokens [B, S] (prompt in [0, P), draft in [P, S))."""
    info = _reduce_draft(W, tokens, prompt_len, decide_bf16)
    new_draft, n_unm, n_edit = edit_rule(tokens[:, prompt_len:], info["top1"], info["conf"], tau, W.shape.mask_id)
    out = tokens.copy()
    out[:, prompt_len:] = new_draft
    info.update({"n_unmasked": n_unm, "n_edited": n_edit})
    return out, info


# ------------------------------------------- two thresholds and the EOS stop

def edit_rule_ex(draft: np.ndarray, top1: np.ndarray, conf: np.ndarray, tau_unmask: float, tau_edit: float,
                 mask_id: int, eos_id: int = -1):
    """Editing rule with separate thresholds (App. C.4 names the native
    token-editing rule and its early end: no confident edit left, or an EOS
    token produced; the reading used here): from one forward, a [MASK] slot
    takes its top-1 when top1 != mask_id and conf >= tau_unmask, a real-token
    slot when top1 != mask_id and conf >= tau_edit.  Also returns how many
    slots were newly set to eos_id (0 when eos_id < 0)."""
    is_mask = draft == mask_id
    thr = np.where(is_mask, tau_unmask, tau_edit)
    take = (top1 != mask_id) & (conf >= thr)
    new = np.where(take, top1, draft).astype(draft.dtype)
    changed = new != draft
    n_unmasked = int(np.sum(changed & is_mask))
    n_edited = int(np.sum(changed & ~is_mask))
    n_eos = int(np.sum(changed & (new == eos_id))) if eos_id >= 0 else 0
    return new, n_unmasked, n_edited, n_eos


def refine_step_ex(W, tokens: np.ndarray, prompt_len: int, tau_unmask: float, tau_edit: float, eos_id: int = -1,
                   decide_bf16: bool = False, span_start: int = 0):
    """One refinement pass under edit_rule_ex.  With span_start, the draft part
    of tokens is a span of a longer draft: its token i sits at position
    prompt_len + span_start + i."""
    S = tokens.shape[1]
    positions = None
    if span_start:
        positions = np.concatenate([np.arange(prompt_len), prompt_len + span_start + np.arange(S - prompt_len)])
    info = _reduce_draft(W, tokens, prompt_len, decide_bf16, positions)
    new_draft, n_unm, n_edit, n_eos = edit_rule_ex(tokens[:, prompt_len:], info["top1"], info["conf"],
                                                   tau_unmask, tau_edit, W.shape.mask_id, eos_id)
    out = tokens.copy()
    out[:, prompt_len:] = new_draft
    info.update({"n_unmasked": n_unm, "n_edited": n_edit, "n_eos": n_eos})
    return out, info


def refine_ex(W, prompt: np.ndarray, draft: np.ndarray, mask: np.ndarray | None, n_steps: int,
              tau_unmask: float, tau_edit: float, eos_id: int = -1, decide_bf16: bool = False):
    """refine() under edit_rule_ex: stops after a pass that changed nothing
    (stop_reason 1) or, with eos_id >= 0, after a pass that wrote eos_id into a
    draft slot (stop_reason 2); 0 when the pass budget ran out."""
    shape = W.shape
    P = prompt.shape[1]
    d = draft.copy()
    if mask is not None:
        d[mask] = shape.mask_id
    tokens = np.concatenate([prompt, d], axis=1).astype(np.int32)
    stats = {"steps_run": 0, "n_unmasked": 0, "n_edited": 0, "stop_reason": 0, "per_step": []}
    for _ in range(n_steps):
        tokens, info = refine_step_ex(W, tokens, P, tau_unmask, tau_edit, eos_id, decide_bf16)
        stats["steps_run"] += 1
        stats["n_unmasked"] += info["n_unmasked"]
        stats["n_edited"] += info["n_edited"]
        stats["per_step"].append(info)
        if info["n_unmasked"] + info["n_edited"] == 0:
            stats["stop_reason"] = 1
            break
        if eos_id >= 0 and info["n_eos"] > 0:
            stats["stop_reason"] = 2
            break
    stats["n_masked_left"] = int(np.sum(tokens[:, P:] == shape.mask_id))
    return tokens[:, P:].copy(), stats


def refine_local(W, prompt: np.ndarray, draft: np.ndarray, mask: np.ndarray | None, schedule,
                 tau_unmask: float, tau_edit: float, eos_id: int = -1, decide_bf16: bool = False):
    """Local / staged refinement (Sec. 6.3 and Table 10: refinement in 64-token
    chunks of the generated span; App. D.4: staged schedules of span sizes).
    Reading used here: for each stage (span, passes) of the schedule, the draft
    is cut into chunks of `span` tokens (the last may be shorter); a chunk is
    refined on its own -- the sequence is prompt ‖ chunk, the chunk's tokens at
    their positions in the full sequence -- for up to `passes` passes of
    refine_step_ex, stopping after a pass that changed nothing in it; a pass
    that writes eos_id (eos_id >= 0) ends the whole run.  stop_reason: 0 some
    chunk used its whole budget, 1 every chunk stopped without change, 2 EOS."""
    shape = W.shape
    P = prompt.shape[1]
    D = draft.shape[1]
    d = draft.copy()
    if mask is not None:
        d[mask] = shape.mask_id
    stats = {"steps_run": 0, "n_unmasked": 0, "n_edited": 0, "stop_reason": 1, "chunks": []}
    eos_stop = False
    for span, passes in schedule:
        L = min(int(span), D)
        for c0 in range(0, D, L):
            if eos_stop:
                break
            tokens = np.concatenate([prompt, d[:, c0:c0 + L]], axis=1).astype(np.int32)
            still = False
            for _ in range(passes):
                tokens, info = refine_step_ex(W, tokens, P, tau_unmask, tau_edit, eos_id, decide_bf16, span_start=c0)
                stats["steps_run"] += 1
                stats["n_unmasked"] += info["n_unmasked"]
                stats["n_edited"] += info["n_edited"]
                if info["n_unmasked"] + info["n_edited"] == 0:
                    still = True
                    break
                if eos_id >= 0 and info["n_eos"] > 0:
                    eos_stop = True
                    break
            if not still and passes > 0 and stats["stop_reason"] != 2:
                stats["stop_reason"] = 0
            d[:, c0:c0 + L] = tokens[:, P:]
            stats["chunks"].append((c0, L))
        if eos_stop:
            break
    if eos_stop:
        stats["stop_reason"] = 2
    stats["n_masked_left"] = int(np.sum(d == shape.mask_id))
    return d, stats


def refine(W, prompt: np.ndarray, draft: np.ndarray, mask: np.ndarray | None, n_steps: int,
           tau: float, decide_bf16: bool = False):
    """Draft positions in the mask set start as [MASK]; then up to n_steps passes,
    stopping after a pass that changed nothing.  Returns (final draft, stats)."""
    shape = W.shape
    P = prompt.shape[1]
    d = draft.copy()
    if mask is not None:
        d[mask] = shape.mask_id
    tokens = np.concatenate([prompt, d], axis=1).astype(np.int32)
    stats = {"steps_run": 0, "n_unmasked": 0, "n_edited": 0, "per_step": []}
    for _ in range(n_steps):
        tokens, info = refine_step(W, tokens, P, tau, decide_bf16)
        stats["steps_run"] += 1
        stats["n_unmasked"] += info["n_unmasked"]
        stats["n_edited"] += info["n_edited"]
        stats["per_step"].append(info)
        if info["n_unmasked"] + info["n_edited"] == 0:
            break
    stats["n_masked_left"] = int(np.sum(tokens[:, P:] == shape.mask_id))
    return tokens[:, P:].copy(), stats
