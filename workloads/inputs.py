"""Seeded prompt/draft token draws and mask-set draws.

The refiner's inputs are a fixed prompt, a complete draft and a set of draft
positions to start as [MASK] (Sec. 4.2; the all-[MASK] variant of Sec. 6.3 is
the special case where the mask set is every draft position).  These helpers
draw such inputs from a seed with NumPy's PCG64; they compute nothing of the
refinement itself.
"""

from __future__ import annotations

import numpy as np

from .configs import Workload


def _zipf_table(n_ranks: int, exponent: float) -> np.ndarray:
    # Cumulative distribution of P(r) proportional to r**-exponent, r = 1..n_ranks.
    r = np.arange(1, n_ranks + 1, dtype=np.float64)
    p = r ** (-exponent)
    cdf = np.cumsum(p)
    return cdf / cdf[-1]


def draw_tokens(rng: np.random.Generator, shape, vocab: int, dist: str = "uniform") -> np.ndarray:
    """Token ids in [0, vocab-2]; the last id (the [MASK] id) is never drawn.

    ``dist="zipf1.1"`` draws rank r in 1..vocab-1 with P(r) ~ r**-1.1 and maps it
    to id r-1, so small ids are frequent (skewed expert load).
    """
    if dist == "uniform":
        return rng.integers(0, vocab - 1, size=shape, dtype=np.int64).astype(np.int32)
    if dist.startswith("zipf"):
        a = float(dist[4:])
        cdf = _zipf_table(vocab - 1, a)
        u = rng.random(size=shape)
        idx = np.searchsorted(cdf, u, side="right")
        return np.minimum(idx, vocab - 2).astype(np.int32)
    raise ValueError(f"unknown token distribution {dist!r}")


def draw_mask_set(rng: np.random.Generator, batch: int, draft_len: int, frac: float) -> np.ndarray:
    """Boolean [batch, draft_len]: exactly floor(frac*draft_len + 1/2) positions per row."""
    n_mask = int(np.floor(frac * draft_len + 0.5))
    m = np.zeros((batch, draft_len), dtype=bool)
    for b in range(batch):
        if n_mask:
            m[b, rng.choice(draft_len, size=n_mask, replace=False)] = True
    return m


def make_inputs(w: Workload, batch: int | None = None, seed: int | None = None):
    """(prompt [B,P] int32, draft [B,D] int32, mask [B,D] bool) for a workload."""
    B = w.batch if batch is None else batch
    rng = np.random.default_rng(w.input_seed if seed is None else seed)
    V = w.model.vocab
    prompt = draw_tokens(rng, (B, w.prompt_len), V, w.token_dist)
    draft = draw_tokens(rng, (B, w.draft_len), V, w.token_dist)
    mask = draw_mask_set(rng, B, w.draft_len, w.mask_frac)
    return prompt, draft, mask
