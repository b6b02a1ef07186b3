"""Hand-built weight sets for oracle pins (closed-form end-to-end cases)."""

from __future__ import annotations

import numpy as np


class PlantedWeights:
    """Duck-typed stand-in for oracle.OracleWeights with explicit arrays."""

    def __init__(self, shape, embed, lm_head, layers, final_norm=None):
        self.shape = shape
        self._embed = np.asarray(embed, dtype=np.float64)
        self._lm = np.asarray(lm_head, dtype=np.float64)
        self._layers = layers
        self._gf = np.ones(shape.d_model) if final_norm is None else np.asarray(final_norm)

    def embed_rows(self, ids):
        return self._embed[np.asarray(ids)]

    def embed(self):
        return self._embed

    def lm_head(self):
        return self._lm

    def final_norm(self):
        return self._gf

    def layer(self, l):
        return self._layers[l]


def zero_block(shape, rng=None, scale=0.05):
    """A layer whose attention output projection and FFN down projection are zero,
    so the block is the identity on the residual stream; the other matrices are
    random so that a wrong residual wiring would show."""
    rng = rng or np.random.default_rng(0)
    d, hd, H, KV = shape.d_model, shape.head_dim, shape.n_heads, shape.n_kv_heads
    r = lambda *s: rng.standard_normal(s) * scale
    L = {"wq": r(H * hd, d), "wk": r(KV * hd, d), "wv": r(KV * hd, d),
         "wo": np.zeros((d, H * hd)), "g1": np.ones(d), "g2": np.ones(d)}
    if shape.n_experts == 0:
        L.update(w_gate=r(shape.ffn_dim, d), w_up=r(shape.ffn_dim, d),
                 w_down=np.zeros((d, shape.ffn_dim)))
    else:
        F = shape.expert_ffn_dim
        L["w_router"] = r(shape.n_experts, d)
        L["experts"] = [(r(F, d), r(F, d), np.zeros((d, F))) for _ in range(shape.n_experts)]
        L["shared"] = [(r(F, d), r(F, d), np.zeros((d, F))) for _ in range(shape.n_shared_experts)]
    return L
