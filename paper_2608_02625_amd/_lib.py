"""ctypes binding of libdlm.so (the C ABI declared in include/dlm.h).

Argument marshalling only: every step of the refinement pass runs in the HIP
kernels of the library.  Importing this module fails loudly when the library
has not been built; there is no fallback implementation.
"""

from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdlm.so")

DLM_OK = 0
STATIC_SCRATCH_BYTES = 64 << 20      # DLM_STATIC_SCRATCH_BYTES of include/dlm.h
STATUS_NAMES = {0: "DLM_OK", -1: "DLM_ERR_INVALID_ARG", -3: "DLM_ERR_HIP", -4: "DLM_ERR_UNSUPPORTED",
                -5: "DLM_ERR_WORKSPACE", -6: "DLM_ERR_NO_MEMORY", -7: "DLM_ERR_INTERNAL"}


class DlmConfig(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
        ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32), ("expert_ffn_dim", ctypes.c_int32),
        ("n_shared_experts", ctypes.c_int32), ("vocab", ctypes.c_int32), ("mask_id", ctypes.c_int32),
        ("rope_theta", ctypes.c_float), ("norm_eps", ctypes.c_float), ("init_std", ctypes.c_float),
        ("lm_head_scale", ctypes.c_float),
    ]


class DlmStats(ctypes.Structure):
    _fields_ = [("n_unmasked", ctypes.c_int32), ("n_edited", ctypes.c_int32),
                ("n_masked_left", ctypes.c_int32), ("steps_run", ctypes.c_int32),
                ("n_invalid", ctypes.c_int32)]

    def as_dict(self):
        return {f: int(getattr(self, f)) for f, _ in self._fields_}


# (name, restype, argtypes) of every entry point in include/dlm.h
class DlmEditRule(ctypes.Structure):
    _fields_ = [("unmask_threshold", ctypes.c_float), ("edit_threshold", ctypes.c_float),
                ("eos_id", ctypes.c_int32)]


class DlmCascadeStats(ctypes.Structure):
    _fields_ = [("draft", DlmStats), ("refine", DlmStats), ("draft_passes", ctypes.c_int32),
                ("refine_passes", ctypes.c_int32), ("refine_stop_reason", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("draft_ms", ctypes.c_double), ("refine_ms", ctypes.c_double)]

    def as_dict(self):
        return {"draft": self.draft.as_dict(), "refine": self.refine.as_dict(),
                "draft_passes": int(self.draft_passes), "refine_passes": int(self.refine_passes),
                "refine_stop_reason": int(self.refine_stop_reason), "draft_ms": float(self.draft_ms),
                "refine_ms": float(self.refine_ms)}


_P = ctypes.c_void_p
_I = ctypes.c_int32
_F = ctypes.c_float
_SZ = ctypes.c_size_t
_CFG = ctypes.POINTER(DlmConfig)
SIGNATURES = [
    ("dlm_weights_bytes", _SZ, [_CFG]),
    ("dlm_workspace_bytes", _SZ, [_CFG, _I, _I, _I]),
    ("dlm_load_synthetic_weights", _I, [_CFG, ctypes.c_uint64, _P, _SZ, _P, ctypes.POINTER(_P)]),
    ("dlm_refine_step", _I, [_P, _I, _I, _I, _P, _F, _P, _SZ, _P, _P, _P, _P]),
    ("dlm_refine_step_static", _I, [_P, _I, _I, _I, _P, _F, _P, _P, _P, _P]),
    ("dlm_refine", _I, [_P, _I, _I, _I, _P, _P, _P, _I, _F, _P, _SZ, _P, ctypes.POINTER(DlmStats)]),
    ("dlm_refine_step_ex", _I, [_P, _I, _I, _I, _P, ctypes.POINTER(DlmEditRule), _P, _SZ, _P, _P, _P, _P, _P]),
    ("dlm_refine_ex", _I, [_P, _I, _I, _I, _P, _P, _P, _I, ctypes.POINTER(DlmEditRule), _P, _SZ, _P,
                           ctypes.POINTER(DlmStats), ctypes.POINTER(_I)]),
    ("dlm_refine_step_span", _I, [_P, _I, _I, _I, _I, _P, ctypes.POINTER(DlmEditRule), _P, _SZ, _P, _P, _P, _P,
                                  _P]),
    ("dlm_refine_local", _I, [_P, _I, _I, _I, _P, _P, _P, _I, _P, _P, ctypes.POINTER(DlmEditRule), _P, _SZ, _P,
                              ctypes.POINTER(DlmStats), ctypes.POINTER(_I)]),
    ("dlm_draft_workspace_bytes", _SZ, [_CFG, _I, _I, _I, _I]),
    ("dlm_draft", _I, [_P, _I, _I, _I, _P, _P, _I, _I, _F, _P, _SZ, _P, ctypes.POINTER(DlmStats),
                       ctypes.POINTER(_I)]),
    ("dlm_draft_step", _I, [_P, _I, _I, _I, _I, _I, _I, _F, _P, _P, _SZ, _P, _P, _P, _P, _P]),
    ("dlm_cascade_workspace_bytes", _SZ, [_CFG, _CFG, _I, _I, _I, _I]),
    ("dlm_cascade", _I, [_P, _P, _I, _I, _I, _P, _P, _I, _I, _F, _I, ctypes.POINTER(DlmEditRule), _P, _SZ, _P,
                         ctypes.POINTER(DlmCascadeStats)]),
    ("dlm_debug_forward", _I, [_P, _I, _I, _I, _P, _P, _SZ, _P, _P, _P, _P, _P, _P, _P, _P]),
    ("dlm_debug_layer", _I, [_P, _I, _I, _I, _P, _P, _P, _SZ, _P, _P, _P]),
    ("dlm_debug_head", _I, [_P, _I, _I, _I, _P, _P, _SZ, _P, _P, _P, _P]),
    ("dlm_debug_gemm", _I, [_P, _P, _P, _I, _I, _I, _I, _I, _P]),
    ("dlm_weight_info", _I, [_P, _I, _I, _I, ctypes.POINTER(_P), ctypes.POINTER(_I)]),
    ("dlm_set_profiling", _I, [_P, ctypes.c_char_p]),
    ("dlm_profile_read", _I, [_P, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(_F), _I]),
    ("dlm_debug_fail_host_alloc", _I, [_I]),
    ("dlm_free", None, [_P]),
    ("dlm_last_error", ctypes.c_char_p, []),
]

_lib = None


def load(path: str = LIB_PATH):
    """Load libdlm.so and attach prototypes; raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build the HIP library first "
            "(python -m paper_2608_02625_amd.build or __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    for name, res, args in SIGNATURES:
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class DlmError(RuntimeError):
    pass


def check(status: int, what: str = ""):
    if status != DLM_OK:
        msg = load().dlm_last_error()
        msg = msg.decode() if msg else ""
        raise DlmError(f"{what}: {STATUS_NAMES.get(status, status)}: {msg}")
