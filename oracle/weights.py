"""Synthetic refiner weights, regenerated on the CPU.

CPU oracle -- test infrastructure only.  Only tests/, the smoke check and the
benchmark's CPU-baseline leg may import this module; the GPU product path never
does, and this module imports nothing from it.

The paper uses public checkpoints (Sec. 5.1) that are not available here, so
the refiner's weights are synthetic: every matrix element is an Irwin-Hall
draw (rng.c) scaled to standard deviation init_std (times lm_head_scale for the
LM head) and rounded to bfloat16:

    c     = float32(init_std * scale * sqrt(3) / 65536)   (computed in float64)
    value = bfloat16_rne(float32(n) * c)                  (one IEEE fp32 multiply)

RMSNorm gains are 1.  Tensors are logical [out_features, in_features] matrices
addressed by a 32-bit id: (layer_field << 20) | (kind << 12) | expert, with
layer_field 0 for the embedding and LM head and l+1 for layer l.

Values are returned as float32 arrays holding exact bfloat16 values; the
oracle's arithmetic upcasts them to float64.
"""

from __future__ import annotations

import ctypes
import math
import os

import numpy as np
import torch

from . import build as _build

# Tensor kinds.
K_EMBED, K_LM_HEAD = 0, 1                     # layer_field 0
K_WQ, K_WK, K_WV, K_WO = 0, 1, 2, 3           # layer_field l+1
K_FFN_GATE, K_FFN_UP, K_FFN_DOWN = 4, 5, 6
K_ROUTER = 7
K_EXP_GATE, K_EXP_UP, K_EXP_DOWN = 8, 9, 10
K_SH_GATE, K_SH_UP, K_SH_DOWN = 11, 12, 13


def tensor_id(layer_field: int, kind: int, expert: int = 0) -> int:
    return (layer_field << 20) | (kind << 12) | expert


_lib = None


def _rng():
    global _lib
    if _lib is None:
        path = _build.build(force=False)
        lib = ctypes.CDLL(path)
        lib.oracle_philox4x32_10.argtypes = [ctypes.POINTER(ctypes.c_uint32)] * 3
        lib.oracle_philox4x32_10.restype = None
        lib.oracle_irwin_hall.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64,
                                          ctypes.c_uint64, ctypes.c_void_p]
        lib.oracle_irwin_hall.restype = None
        lib.oracle_irwin_hall_at.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p,
                                             ctypes.c_uint64, ctypes.c_void_p]
        lib.oracle_irwin_hall_at.restype = None
        _lib = lib
    return _lib


def philox4x32_10(ctr, key):
    """One Philox4x32-10 block: 4 counter words, 2 key words -> 4 output words."""
    c = (ctypes.c_uint32 * 4)(*[int(x) & 0xffffffff for x in ctr])
    k = (ctypes.c_uint32 * 2)(*[int(x) & 0xffffffff for x in key])
    o = (ctypes.c_uint32 * 4)()
    _rng().oracle_philox4x32_10(c, k, o)
    return [int(x) for x in o]


def irwin_hall(seed: int, tid: int, start: int, count: int) -> np.ndarray:
    out = np.empty(count, dtype=np.int32)
    if count:
        _rng().oracle_irwin_hall(seed, tid, start, count, out.ctypes.data)
    return out


def irwin_hall_at(seed: int, tid: int, idx: np.ndarray) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.uint64)
    out = np.empty(idx.size, dtype=np.int32)
    if idx.size:
        _rng().oracle_irwin_hall_at(seed, tid, idx.ctypes.data, idx.size, out.ctypes.data)
    return out


def scale_constant(init_std: float, scale: float = 1.0) -> np.float32:
    return np.float32(init_std * scale * math.sqrt(3.0) / 65536.0)


def to_weight_values(n: np.ndarray, c: np.float32) -> np.ndarray:
    """float32(n) * c in IEEE fp32, then round-to-nearest-even to bfloat16 (torch)."""
    prod = n.astype(np.float32) * np.float32(c)
    bf = torch.from_numpy(prod).to(torch.bfloat16)
    return bf.to(torch.float32).numpy()


def weight_matrix(seed: int, tid: int, rows: int, cols: int, init_std: float,
                  scale: float = 1.0, row_start: int = 0, row_count: int | None = None) -> np.ndarray:
    """Rows [row_start, row_start+row_count) of a logical [rows, cols] matrix, float32."""
    if row_count is None:
        row_count = rows - row_start
    n = irwin_hall(seed, tid, row_start * cols, row_count * cols)
    return to_weight_values(n, scale_constant(init_std, scale)).reshape(row_count, cols)


def weight_values_at(seed: int, tid: int, idx: np.ndarray, init_std: float, scale: float = 1.0):
    """Values of the given flat element indices of one tensor, float32."""
    return to_weight_values(irwin_hall_at(seed, tid, idx), scale_constant(init_std, scale))


class _Experts:
    """Expert (gate, up, down) weight triples generated when indexed (the
    flash-scale slice has 256 experts of 19M weights each per layer)."""

    def __init__(self, make, n: int, cache: bool):
        self._make, self._n = make, n
        self._cache = {} if cache else None

    def __len__(self):
        return self._n

    def __getitem__(self, e: int):
        if not 0 <= e < self._n:
            raise IndexError(e)
        if self._cache is None:
            return self._make(e)
        if e not in self._cache:
            self._cache[e] = self._make(e)
        return self._cache[e]


class OracleWeights:
    """Lazily regenerated refiner weights for one (shape, seed)."""

    def __init__(self, shape, seed: int, cache_layers: bool = True):
        self.shape = shape
        self.seed = int(seed)
        self.cache_layers = cache_layers
        self._layers = {}
        self._embed = None
        self._lm_head = None

    # -- global tensors -------------------------------------------------
    def embed(self) -> np.ndarray:
        s = self.shape
        if self._embed is None:
            self._embed = weight_matrix(self.seed, tensor_id(0, K_EMBED), s.vocab, s.d_model,
                                        s.init_std)
        return self._embed

    def embed_rows(self, token_ids: np.ndarray) -> np.ndarray:
        """Embedding rows for the given ids without materialising the whole table."""
        s = self.shape
        if self._embed is not None:
            return self._embed[token_ids]
        ids = np.asarray(token_ids).reshape(-1).astype(np.uint64)
        idx = (ids[:, None] * np.uint64(s.d_model) + np.arange(s.d_model, dtype=np.uint64)[None, :])
        vals = weight_values_at(self.seed, tensor_id(0, K_EMBED), idx.reshape(-1), s.init_std)
        return vals.reshape(*np.asarray(token_ids).shape, s.d_model)

    def lm_head(self) -> np.ndarray:
        s = self.shape
        if self._lm_head is None:
            self._lm_head = weight_matrix(self.seed, tensor_id(0, K_LM_HEAD), s.vocab, s.d_model,
                                          s.init_std, s.lm_head_scale)
        return self._lm_head

    def final_norm(self) -> np.ndarray:
        return np.ones(self.shape.d_model, dtype=np.float32)

    # -- per-layer tensors ------------------------------------------------
    def layer(self, l: int) -> dict:
        if l in self._layers:
            return self._layers[l]
        s = self.shape
        f = l + 1
        m = lambda kind, rows, cols, e=0: weight_matrix(self.seed, tensor_id(f, kind, e), rows, cols,
                                                       s.init_std)
        d, hd = s.d_model, s.head_dim
        L = {
            "wq": m(K_WQ, s.n_heads * hd, d),
            "wk": m(K_WK, s.n_kv_heads * hd, d),
            "wv": m(K_WV, s.n_kv_heads * hd, d),
            "wo": m(K_WO, d, s.n_heads * hd),
            "g1": np.ones(d, dtype=np.float32),
            "g2": np.ones(d, dtype=np.float32),
        }
        if s.n_experts == 0:
            L["w_gate"] = m(K_FFN_GATE, s.ffn_dim, d)
            L["w_up"] = m(K_FFN_UP, s.ffn_dim, d)
            L["w_down"] = m(K_FFN_DOWN, d, s.ffn_dim)
        else:
            F = s.expert_ffn_dim
            L["w_router"] = m(K_ROUTER, s.n_experts, d)
            L["experts"] = _Experts(
                lambda e: (m(K_EXP_GATE, F, d, e), m(K_EXP_UP, F, d, e), m(K_EXP_DOWN, d, F, e)),
                s.n_experts, self.cache_layers)
            L["shared"] = [
                (m(K_SH_GATE, F, d, e), m(K_SH_UP, F, d, e), m(K_SH_DOWN, d, F, e))
                for e in range(s.n_shared_experts)
            ]
        if self.cache_layers:
            self._layers[l] = L
        return L
