"""Plain float64 CPU implementation of block-autoregressive drafting.

CPU oracle -- test infrastructure only.  Only tests/, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with the
GPU library and imports nothing from it.

What is computed (paper: Sec. 3.3 "Block Autoregressive Diffusion", Sec. 4.1
"Drafting"; Table 9 and Table 10 for the b/s/t draft settings):

  * The response of draft_len positions is split into blocks of block_len
    positions (the last one may be shorter).  Blocks are generated in order;
    each starts all [MASK] and is denoised by up to T_d steps.
  * Visibility is block-causal (Sec. 3.3): a position of block k attends to the
    prompt, to blocks 0..k-1 and bidirectionally to its own block, never to a
    later block.  The prompt is read as one unit that attends to itself only
    (reading: the paper conditions every block on x and says no more).
    A step on block k is therefore one forward over positions [0, end of block
    k) with that mask; later positions cannot influence it.
  * Unmasking (reading of the b/s/t triple, Table 9 and Table 10: block size,
    steps per block, confidence threshold): with n masked slots left in the
    block and r steps left for it, the step's quota is ceil(n / r).  Every
    masked slot whose top-1 confidence is >= t is unmasked; when that is fewer
    than the quota, the quota most confident masked slots are unmasked
    instead (equal confidences: lower position first).  An unmasked slot
    takes its top-1 token and keeps it (drafting does not edit).  A block ends
    once it holds no [MASK], at the latest after T_d steps, so it costs at most
    T_d passes (the K x T_d cost of Sec. 4.1).
  * Batches: all sequences share the block positions; a step runs over the
    whole batch and changes only sequences that still have masked slots in the
    block; the block ends when none has.
  * Speculative correction (Sec. 4.3): a drafter drafts, a refiner (sharing the
    vocabulary) refines the finished draft; the cost is K x T_d drafting passes
    plus T_r refinement passes (Sec. 4.2).
"""

from __future__ import annotations

import numpy as np

from .refine import forward, lm_head_reduce, refine_ex


def block_key_limit(prompt_len: int, seq_len: int, block_len: int) -> np.ndarray:
    """Per position, how many leading keys it may attend to under block-causal
    visibility: the prompt sees the prompt; block j (positions prompt_len +
    j*block_len ...) sees everything up to the end of block j."""
    pos = np.arange(seq_len)
    blk = (pos - prompt_len) // block_len
    lim = np.where(pos < prompt_len, prompt_len, prompt_len + (blk + 1) * block_len)
    return np.minimum(lim, seq_len)


def draft_select(is_mask: np.ndarray, conf: np.ndarray, tau: float, steps_left: int) -> np.ndarray:
    """The slots of one block a drafting step unmasks.

    is_mask, conf: [B, n] for the n slots of the block.  Per sequence: quota =
    ceil(#masked / steps_left); take every masked slot with conf >= tau, or, if
    those are fewer than the quota, the quota masked slots of highest
    confidence (ties to the lower position).
    """
    B, n = is_mask.shape
    sel = np.zeros((B, n), dtype=bool)
    for b in range(B):
        masked = [i for i in range(n) if is_mask[b, i]]
        if not masked:
            continue
        quota = -(-len(masked) // steps_left)
        n_above = sum(1 for i in masked if conf[b, i] >= tau)
        order = sorted(masked, key=lambda i: (-float(conf[b, i]), i))
        for i in order[:max(quota, n_above)]:
            sel[b, i] = True
    return sel


def block_bounds(prompt_len: int, draft_len: int, block_len: int, k: int):
    start = prompt_len + k * block_len
    return start, min(start + block_len, prompt_len + draft_len)


def draft_forward_block(W, tokens: np.ndarray, prompt_len: int, block_len: int, k: int, decide_bf16: bool = False):
    """Forward over the prefix that ends with block k under the block-causal
    mask; top-1, confidence and logit statistics of block k's positions."""
    B, S = tokens.shape
    start, end = block_bounds(prompt_len, S - prompt_len, block_len, k)
    x = forward(W, tokens[:, :end], decide_bf16=decide_bf16,
                key_limit=block_key_limit(prompt_len, end, block_len))
    n = end - start
    red = lm_head_reduce(W, x[:, start:end].reshape(B * n, -1), decide_bf16=decide_bf16)
    return {key: red[key].reshape(B, n) for key in ("top1", "conf", "max_logit", "margin")}


def draft_step(W, tokens: np.ndarray, prompt_len: int, block_len: int, k: int, tau: float, steps_left: int,
               decide_bf16: bool = False):
    """One denoising step on block k of tokens [B, S]: returns the new tokens
    and the step's info (top1, conf, margin of the block, sel, n_unmasked)."""
    start, end = block_bounds(prompt_len, tokens.shape[1] - prompt_len, block_len, k)
    info = draft_forward_block(W, tokens, prompt_len, block_len, k, decide_bf16)
    cur = tokens[:, start:end]
    sel = draft_select(cur == W.shape.mask_id, info["conf"], tau, steps_left)
    out = tokens.copy()
    out[:, start:end] = np.where(sel, info["top1"], cur)
    info["sel"] = sel
    info["n_unmasked"] = int(np.sum(out[:, start:end] != cur))
    return out, info


def draft(W, prompt: np.ndarray, draft_len: int, block_len: int, steps: int, tau: float,
          decide_bf16: bool = False):
    """Block-AR drafting of draft_len tokens after prompt [B, P].

    Returns (draft [B, draft_len], stats) with stats = {"steps_run": passes
    over all blocks, "block_steps": passes per block, "n_masked_left"}.
    """
    prompt = np.asarray(prompt)
    B, P = prompt.shape
    mask_id = W.shape.mask_id
    tokens = np.concatenate([prompt, np.full((B, draft_len), mask_id, dtype=prompt.dtype)], axis=1)
    n_blocks = -(-draft_len // block_len)
    block_steps = []
    for k in range(n_blocks):
        start, end = block_bounds(P, draft_len, block_len, k)
        used = 0
        for t in range(steps):
            if not np.any(tokens[:, start:end] == mask_id):
                break
            tokens, _ = draft_step(W, tokens, P, block_len, k, tau, steps - t, decide_bf16)
            used += 1
        block_steps.append(used)
    out = tokens[:, P:]
    return out, {"steps_run": int(sum(block_steps)), "block_steps": block_steps,
                 "n_masked_left": int(np.sum(out == mask_id))}


def cascade(W_draft, W_refine, prompt: np.ndarray, draft_len: int, block_len: int, steps: int, tau_draft: float,
            n_refine: int, tau_unmask: float, tau_edit: float, eos_id: int = -1, decide_bf16: bool = False):
    """Draft with W_draft, then refine_ex with W_refine on the finished draft
    (no mask set).  Returns (refined draft, {"draft", "refine", "passes"})."""
    d, ds = draft(W_draft, prompt, draft_len, block_len, steps, tau_draft, decide_bf16)
    r, rs = refine_ex(W_refine, prompt, d, None, n_refine, tau_unmask, tau_edit, eos_id, decide_bf16)
    return r, {"draft": ds, "refine": rs, "draft_tokens": d, "passes": ds["steps_run"] + rs["steps_run"]}
