"""Python front end of the refinement-step library.

PyTorch supplies device memory and the stream; every computation of the
refinement pass runs in libdlm.so's HIP kernels through the C ABI.
"""

from __future__ import annotations

import ctypes

import torch

from . import _lib
from ._lib import DlmConfig, DlmStats, check

CONFIG_FIELDS = [f for f, _ in DlmConfig._fields_]


def make_config(shape) -> DlmConfig:
    """DlmConfig from a mapping or an object with the dlm_config field names."""
    get = (lambda k: shape[k]) if isinstance(shape, dict) else (lambda k: getattr(shape, k))
    cfg = DlmConfig()
    for f in CONFIG_FIELDS:
        setattr(cfg, f, get(f))
    return cfg


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


class Refiner:
    """A refiner with synthetic weights resident in HBM.

    shape: mapping/object with the dlm_config fields; seed: weight seed.
    """

    def __init__(self, shape, seed: int, device: str | torch.device = "cuda"):
        self.lib = _lib.load()
        self.device = torch.device(device)
        self.cfg = make_config(shape)
        nbytes = self.lib.dlm_weights_bytes(ctypes.byref(self.cfg))
        if nbytes == 0:
            raise ValueError("invalid refiner shape")
        self.weights = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self._handle = ctypes.c_void_p()
        check(self.lib.dlm_load_synthetic_weights(ctypes.byref(self.cfg), int(seed), self.weights.data_ptr(),
                                                  nbytes, self.stream, ctypes.byref(self._handle)),
              "dlm_load_synthetic_weights")
        self._ws = {}

    # -------------------------------------------------------------- plumbing
    @property
    def stream(self) -> int:
        return torch.cuda.current_stream(self.device).cuda_stream

    @property
    def mask_id(self) -> int:
        return int(self.cfg.mask_id)

    def workspace(self, batch: int, prompt_len: int, draft_len: int) -> torch.Tensor:
        key = (batch, prompt_len, draft_len)
        ws = self._ws.get(key)
        if ws is None:
            n = self.lib.dlm_workspace_bytes(ctypes.byref(self.cfg), batch, prompt_len, draft_len)
            if n == 0:
                raise ValueError(f"invalid shape {key}")
            ws = torch.empty(n, dtype=torch.uint8, device=self.device)
            self._ws[key] = ws
        return ws

    def close(self):
        if getattr(self, "_handle", None) and self._handle.value:
            self.lib.dlm_free(self._handle)
            self._handle = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -------------------------------------------------------------- refinement
    def refine_step(self, tokens: torch.Tensor, prompt_len: int, threshold: float,
                    top1: torch.Tensor | None = None, conf: torch.Tensor | None = None,
                    stats: torch.Tensor | None = None):
        """One pass over tokens (int32 [B, S], updated in place)."""
        B, S = tokens.shape
        D = S - prompt_len
        ws = self.workspace(B, prompt_len, D)
        check(self.lib.dlm_refine_step(self._handle, B, prompt_len, D, tokens.data_ptr(), float(threshold),
                                       ws.data_ptr(), ws.numel(), self.stream, _ptr(top1), _ptr(conf),
                                       _ptr(stats)), "dlm_refine_step")
        return tokens

    def refine_step_static(self, tokens: torch.Tensor, prompt_len: int, threshold: float,
                           top1: torch.Tensor | None = None, conf: torch.Tensor | None = None,
                           stats: torch.Tensor | None = None):
        """refine_step with the library's static scratch instead of a workspace
        (dlm_refine_step_static: the call allocates nothing)."""
        B, S = tokens.shape
        D = S - prompt_len
        check(self.lib.dlm_refine_step_static(self._handle, B, prompt_len, D, tokens.data_ptr(), float(threshold),
                                              self.stream, _ptr(top1), _ptr(conf), _ptr(stats)),
              "dlm_refine_step_static")
        return tokens

    def refine(self, prompt: torch.Tensor, draft: torch.Tensor, mask: torch.Tensor | None, n_steps: int,
               threshold: float):
        """Refine draft (int32 [B, D], in place) given prompt [B, P] and mask (uint8/bool [B, D])."""
        B, P = prompt.shape
        D = draft.shape[1]
        ws = self.workspace(B, P, D)
        m = None
        if mask is not None:
            m = mask.to(torch.uint8).contiguous()
        st = DlmStats()
        check(self.lib.dlm_refine(self._handle, B, P, D, prompt.data_ptr() if P else None, draft.data_ptr(),
                                  _ptr(m), int(n_steps), float(threshold), ws.data_ptr(), ws.numel(), self.stream,
                                  ctypes.byref(st)), "dlm_refine")
        return draft, st.as_dict()

    def refine_step_ex(self, tokens: torch.Tensor, prompt_len: int, unmask_threshold: float,
                       edit_threshold: float, eos_id: int = -1, top1: torch.Tensor | None = None,
                       conf: torch.Tensor | None = None, stats: torch.Tensor | None = None,
                       eos_written: torch.Tensor | None = None):
        """One pass under the two-threshold rule (tokens int32 [B, S], updated in place)."""
        B, S = tokens.shape
        D = S - prompt_len
        ws = self.workspace(B, prompt_len, D)
        rule = _lib.DlmEditRule(float(unmask_threshold), float(edit_threshold), int(eos_id))
        check(self.lib.dlm_refine_step_ex(self._handle, B, prompt_len, D, tokens.data_ptr(), ctypes.byref(rule),
                                          ws.data_ptr(), ws.numel(), self.stream, _ptr(top1), _ptr(conf),
                                          _ptr(stats), _ptr(eos_written)), "dlm_refine_step_ex")
        return tokens

    def refine_ex(self, prompt: torch.Tensor, draft: torch.Tensor, mask: torch.Tensor | None, n_steps: int,
                  unmask_threshold: float, edit_threshold: float, eos_id: int = -1):
        """refine() under the two-threshold rule with the EOS stop; the stats
        gain stop_reason (0 budget, 1 no change, 2 EOS written)."""
        B, P = prompt.shape
        D = draft.shape[1]
        ws = self.workspace(B, P, D)
        m = None
        if mask is not None:
            m = mask.to(torch.uint8).contiguous()
        st = DlmStats()
        reason = ctypes.c_int32(-1)
        rule = _lib.DlmEditRule(float(unmask_threshold), float(edit_threshold), int(eos_id))
        check(self.lib.dlm_refine_ex(self._handle, B, P, D, prompt.data_ptr() if P else None, draft.data_ptr(),
                                     _ptr(m), int(n_steps), ctypes.byref(rule), ws.data_ptr(), ws.numel(),
                                     self.stream, ctypes.byref(st), ctypes.byref(reason)), "dlm_refine_ex")
        out = st.as_dict()
        out["stop_reason"] = int(reason.value)
        return draft, out

    def refine_step_span(self, tokens: torch.Tensor, prompt_len: int, span_start: int, unmask_threshold: float,
                         edit_threshold: float, eos_id: int = -1, workspace_draft_len: int | None = None,
                         top1: torch.Tensor | None = None, conf: torch.Tensor | None = None,
                         stats: torch.Tensor | None = None, eos_written: torch.Tensor | None = None):
        """One pass over prompt ‖ span (int32 [B, P + L], in place), span token i at position P + span_start + i."""
        B, S = tokens.shape
        L = S - prompt_len
        ws = self.workspace(B, prompt_len, L if workspace_draft_len is None else workspace_draft_len)
        rule = _lib.DlmEditRule(float(unmask_threshold), float(edit_threshold), int(eos_id))
        check(self.lib.dlm_refine_step_span(self._handle, B, prompt_len, L, int(span_start), tokens.data_ptr(),
                                            ctypes.byref(rule), ws.data_ptr(), ws.numel(), self.stream, _ptr(top1),
                                            _ptr(conf), _ptr(stats), _ptr(eos_written)), "dlm_refine_step_span")
        return tokens

    def refine_local(self, prompt: torch.Tensor, draft: torch.Tensor, mask: torch.Tensor | None,
                     schedule: list[tuple[int, int]], unmask_threshold: float, edit_threshold: float,
                     eos_id: int = -1):
        """Local / staged refinement: schedule = [(span, passes), ...] (draft int32 [B, D], in place)."""
        B, P = prompt.shape
        D = draft.shape[1]
        ws = self.workspace(B, P, D)
        m = None
        if mask is not None:
            m = mask.to(torch.uint8).contiguous()
        n = len(schedule)
        spans = (ctypes.c_int32 * max(n, 1))(*[int(a) for a, _ in schedule])
        passes = (ctypes.c_int32 * max(n, 1))(*[int(b) for _, b in schedule])
        st = DlmStats()
        reason = ctypes.c_int32(-1)
        rule = _lib.DlmEditRule(float(unmask_threshold), float(edit_threshold), int(eos_id))
        check(self.lib.dlm_refine_local(self._handle, B, P, D, prompt.data_ptr() if P else None, draft.data_ptr(),
                                        _ptr(m), n, ctypes.cast(spans, ctypes.c_void_p),
                                        ctypes.cast(passes, ctypes.c_void_p), ctypes.byref(rule), ws.data_ptr(),
                                        ws.numel(), self.stream, ctypes.byref(st), ctypes.byref(reason)),
              "dlm_refine_local")
        out = st.as_dict()
        out["stop_reason"] = int(reason.value)
        return draft, out

    # -------------------------------------------------------------- test hooks
    # ------------------------------------------------------- block-AR drafting
    def draft_workspace(self, batch: int, prompt_len: int, draft_len: int, block_len: int) -> torch.Tensor:
        key = ("draft", batch, prompt_len, draft_len, block_len)
        ws = self._ws.get(key)
        if ws is None:
            n = self.lib.dlm_draft_workspace_bytes(ctypes.byref(self.cfg), batch, prompt_len, draft_len, block_len)
            if n == 0:
                raise ValueError(f"invalid drafting shape {key[1:]}")
            ws = torch.empty(n, dtype=torch.uint8, device=self.device)
            self._ws[key] = ws
        return ws

    def draft(self, prompt: torch.Tensor, draft_len: int, block_len: int, steps_per_block: int,
              threshold: float):
        """Block-AR draft of draft_len tokens after prompt [B, P] (int32, on the
        device).  Returns (draft [B, draft_len] int32, stats dict with
        block_steps)."""
        B, P = prompt.shape
        ws = self.draft_workspace(B, P, draft_len, block_len)
        out = torch.empty(B, draft_len, dtype=torch.int32, device=self.device)
        st = DlmStats()
        n_blocks = -(-draft_len // block_len)
        steps = (ctypes.c_int32 * n_blocks)()
        check(self.lib.dlm_draft(self._handle, B, P, draft_len, _ptr(prompt) if P else None, out.data_ptr(),
                                 block_len, steps_per_block, float(threshold), ws.data_ptr(), ws.numel(),
                                 self.stream, ctypes.byref(st), steps), "dlm_draft")
        d = st.as_dict()
        d["block_steps"] = list(steps)
        return out, d

    def draft_step(self, tokens: torch.Tensor, prompt_len: int, block_len: int, block_index: int,
                   steps_left: int, threshold: float, top1: torch.Tensor | None = None,
                   conf: torch.Tensor | None = None, stats: torch.Tensor | None = None,
                   max_logit: torch.Tensor | None = None):
        """One drafting step on block block_index of tokens [B, P + D] (in place)."""
        B, S = tokens.shape
        D = S - prompt_len
        ws = self.draft_workspace(B, prompt_len, D, block_len)
        check(self.lib.dlm_draft_step(self._handle, B, prompt_len, D, block_len, block_index, steps_left,
                                      float(threshold), tokens.data_ptr(), ws.data_ptr(), ws.numel(), self.stream,
                                      _ptr(top1), _ptr(conf), _ptr(max_logit), _ptr(stats)), "dlm_draft_step")
        return tokens

    def debug_forward(self, tokens: torch.Tensor, prompt_len: int, want_logits: bool = False,
                      want_routes: bool = False):
        B, S = tokens.shape
        D = S - prompt_len
        ws = self.workspace(B, prompt_len, D)
        dev = self.device
        hidden = torch.empty(B * S, self.cfg.d_model, dtype=torch.float32, device=dev)
        mx = torch.empty(B * D, dtype=torch.float32, device=dev)
        t1 = torch.empty(B * D, dtype=torch.int32, device=dev)
        cf = torch.empty(B * D, dtype=torch.float32, device=dev)
        lg = torch.empty(B * D, self.cfg.vocab, dtype=torch.float32, device=dev) if want_logits else None
        moe = want_routes and self.cfg.n_experts > 0
        rt = torch.empty(self.cfg.n_layers, B * S, self.cfg.top_k, dtype=torch.int32, device=dev) if moe else None
        rz = torch.empty(self.cfg.n_layers, B * S, self.cfg.n_experts, dtype=torch.float32, device=dev) if moe else None
        check(self.lib.dlm_debug_forward(self._handle, B, prompt_len, D, tokens.data_ptr(), ws.data_ptr(),
                                         ws.numel(), self.stream, hidden.data_ptr(), mx.data_ptr(), t1.data_ptr(),
                                         cf.data_ptr(), _ptr(lg), _ptr(rt), _ptr(rz)), "dlm_debug_forward")
        out = {"hidden": hidden, "max_logit": mx, "top1": t1, "conf": cf}
        if want_logits:
            out["logits"] = lg
        if moe:
            out["routes"] = rt          # [n_layers, B*S, top_k] selected experts per block
            out["router_logits"] = rz   # [n_layers, B*S, n_experts]
        return out

    def debug_layer(self, layer: int, x: torch.Tensor, batch: int, seq_len: int, want_routes: bool = False,
                    want_router_logits: bool = False):
        """One block on the float residual stream x [batch*seq_len, d]; returns the new
        stream, or (stream, expert ids [batch*seq_len, top_k]) with want_routes, or
        (stream, ids, router logits [batch*seq_len, n_experts]) with want_router_logits."""
        ws = self.workspace(batch, 0, seq_len)
        y = torch.empty_like(x)
        ids = z = None
        if (want_routes or want_router_logits) and self.cfg.n_experts > 0:
            ids = torch.empty(batch * seq_len, self.cfg.top_k, dtype=torch.int32, device=self.device)
        if want_router_logits and self.cfg.n_experts > 0:
            z = torch.empty(batch * seq_len, self.cfg.n_experts, dtype=torch.float32, device=self.device)
        check(self.lib.dlm_debug_layer(self._handle, layer, batch, seq_len, x.data_ptr(), y.data_ptr(),
                                       ws.data_ptr(), ws.numel(), self.stream, _ptr(ids), _ptr(z)),
              "dlm_debug_layer")
        if want_router_logits:
            return y, ids, z
        return (y, ids) if want_routes else y

    def debug_head(self, x: torch.Tensor, batch: int, prompt_len: int, draft_len: int):
        ws = self.workspace(batch, prompt_len, draft_len)
        R = batch * draft_len
        mx = torch.empty(R, dtype=torch.float32, device=self.device)
        t1 = torch.empty(R, dtype=torch.int32, device=self.device)
        cf = torch.empty(R, dtype=torch.float32, device=self.device)
        check(self.lib.dlm_debug_head(self._handle, batch, prompt_len, draft_len, x.data_ptr(), ws.data_ptr(),
                                      ws.numel(), self.stream, mx.data_ptr(), t1.data_ptr(), cf.data_ptr()),
              "dlm_debug_head")
        return {"max_logit": mx, "top1": t1, "conf": cf}

    def weight_storage(self, layer_field: int, kind: int, expert: int = 0):
        """(byte offset into self.weights, layout code) of one logical tensor."""
        p = ctypes.c_void_p()
        layout = ctypes.c_int32()
        check(self.lib.dlm_weight_info(self._handle, layer_field, kind, expert, ctypes.byref(p),
                                       ctypes.byref(layout)), "dlm_weight_info")
        return p.value - self.weights.data_ptr(), layout.value

    # -------------------------------------------------------------- profiling
    def set_profiling(self, name_filter: str | None):
        f = None if name_filter is None else name_filter.encode()
        check(self.lib.dlm_set_profiling(self._handle, f), "dlm_set_profiling")

    def profile_read(self, max_entries: int = 1 << 16):
        names = (ctypes.c_char_p * max_entries)()
        ms = (ctypes.c_float * max_entries)()
        n = self.lib.dlm_profile_read(self._handle, names, ms, max_entries)
        if n < 0:
            raise _lib.DlmError("dlm_profile_read failed")
        return [(names[i].decode(), float(ms[i])) for i in range(n)]


# ------------------------------------------------------------------ cascade

_CASCADE_WS = {}


def cascade(drafter: "Refiner", refiner: "Refiner", prompt: torch.Tensor, draft_len: int, block_len: int,
            steps_per_block: int, draft_threshold: float, n_refine_steps: int, unmask_threshold: float,
            edit_threshold: float, eos_id: int = -1):
    """Draft with `drafter`, refine with `refiner` (dlm_cascade).  Returns
    (refined draft [B, draft_len] int32, stats dict)."""
    B, P = prompt.shape
    key = (id(drafter), id(refiner), B, P, draft_len, block_len)
    ws = _CASCADE_WS.get(key)
    if ws is None:
        n = refiner.lib.dlm_cascade_workspace_bytes(ctypes.byref(drafter.cfg), ctypes.byref(refiner.cfg), B, P,
                                                    draft_len, block_len)
        if n == 0:
            raise ValueError(f"invalid cascade shape {key[2:]}")
        ws = torch.empty(n, dtype=torch.uint8, device=refiner.device)
        _CASCADE_WS[key] = ws
    out = torch.empty(B, draft_len, dtype=torch.int32, device=refiner.device)
    rule = _lib.DlmEditRule(float(unmask_threshold), float(edit_threshold), int(eos_id))
    st = _lib.DlmCascadeStats()
    check(refiner.lib.dlm_cascade(drafter._handle, refiner._handle, B, P, draft_len, _ptr(prompt) if P else None,
                                  out.data_ptr(), block_len, steps_per_block, float(draft_threshold),
                                  n_refine_steps, ctypes.byref(rule), ws.data_ptr(), ws.numel(), refiner.stream,
                                  ctypes.byref(st)), "dlm_cascade")
    return out, st.as_dict()


# ------------------------------------------------------------------ GEMM hook

def debug_gemm(a: torch.Tensor, b: torch.Tensor, tile=(256, 256)) -> torch.Tensor:
    """float32 a @ b.T through the library's bf16 MFMA GEMM (a [m,k], b [n,k] bf16)."""
    lib = _lib.load()
    m, k = a.shape
    n = b.shape[0]
    c = torch.empty(m, n, dtype=torch.float32, device=a.device)
    check(lib.dlm_debug_gemm(a.data_ptr(), b.data_ptr(), c.data_ptr(), m, n, k, tile[0], tile[1],
                             torch.cuda.current_stream(a.device).cuda_stream), "dlm_debug_gemm")
    return c
