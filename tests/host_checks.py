"""Host-path checks that test_host_sanitizers.py runs in a child process with a
sanitizer runtime preloaded (not collected by pytest itself).

    host_checks.py abi LIBDLM          the C ABI's validation, planning and error
                                       paths (no GPU work is launched)
    host_checks.py oracle LIBRNG KAT   the oracle's Philox generator against the
                                       published known answers

Prints "host checks passed" at the end; any failed check raises.
"""

from __future__ import annotations

import ctypes
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def _cfg(L, shape, **over):
    d = shape.as_dict()
    d.update(over)
    cfg = L.DlmConfig()
    for f, _ in L.DlmConfig._fields_:
        setattr(cfg, f, d[f])
    return cfg


def abi(path: str) -> None:
    from paper_2608_02625_amd import _lib as L
    from workloads.configs import MODELS

    L.LIB_PATH = path
    lib = L.load(path)
    for name, shape in MODELS.items():
        cfg = _cfg(L, shape)
        wb = lib.dlm_weights_bytes(ctypes.byref(cfg))
        assert wb > 0, name
        assert lib.dlm_workspace_bytes(ctypes.byref(cfg), 2, 64, 64) > 0, name
        assert lib.dlm_draft_workspace_bytes(ctypes.byref(cfg), 2, 64, 128, 64) > 0, name
        # size and shape errors
        assert lib.dlm_workspace_bytes(ctypes.byref(cfg), 0, 64, 64) == 0
        assert lib.dlm_workspace_bytes(ctypes.byref(cfg), 2, -1, 64) == 0
        assert lib.dlm_workspace_bytes(ctypes.byref(cfg), 1 << 20, 1 << 20, 1 << 20) == 0
        assert lib.dlm_draft_workspace_bytes(ctypes.byref(cfg), 2, 64, 128, 0) == 0
        # every load error path before any GPU work
        h = ctypes.c_void_p(1)
        assert lib.dlm_load_synthetic_weights(ctypes.byref(cfg), 0, None, wb, None, ctypes.byref(h)) == -1
        assert h.value is None
        assert lib.dlm_load_synthetic_weights(ctypes.byref(cfg), 0, ctypes.c_void_p(8), wb, None,
                                              ctypes.byref(h)) == -1
        assert b"aligned" in lib.dlm_last_error()
        assert lib.dlm_load_synthetic_weights(ctypes.byref(cfg), 0, ctypes.c_void_p(256), wb - 1, None,
                                              ctypes.byref(h)) == -5
        assert lib.dlm_load_synthetic_weights(ctypes.byref(cfg), 0, ctypes.c_void_p(256), wb, None, None) == -1
    shape = MODELS["mini_moe"]
    for bad in (dict(head_dim=96), dict(top_k=9), dict(mask_id=157184), dict(n_heads=15), dict(n_layers=-1),
                dict(expert_ffn_dim=100), dict(n_experts=300), dict(vocab=1), dict(d_model=-64),
                dict(norm_eps=float("nan")), dict(rope_theta=-1.0), dict(n_kv_heads=0)):
        cfg = _cfg(L, shape, **bad)
        assert lib.dlm_weights_bytes(ctypes.byref(cfg)) == 0, bad
        h = ctypes.c_void_p()
        assert lib.dlm_load_synthetic_weights(ctypes.byref(cfg), 0, ctypes.c_void_p(256), 1 << 40, None,
                                              ctypes.byref(h)) == -1, bad
        assert len(lib.dlm_last_error()) > 0
    assert lib.dlm_weights_bytes(None) == 0
    # entry points with no model
    assert lib.dlm_refine_step(None, 1, 1, 1, None, 0.5, None, 0, None, None, None, None) == -1
    assert lib.dlm_refine_step_static(None, 1, 1, 1, None, 0.5, None, None, None, None) == -1
    assert lib.dlm_refine(None, 1, 1, 1, None, None, None, 1, 0.5, None, 0, None, None) == -1
    assert lib.dlm_draft(None, 1, 1, 64, None, None, 64, 16, 0.25, None, 0, None, None, None) == -1
    assert lib.dlm_draft_step(None, 1, 1, 64, 64, 0, 16, 0.25, None, None, 0, None, None, None, None, None) == -1
    assert lib.dlm_set_profiling(None, None) == -1
    assert lib.dlm_profile_read(None, None, None, 0) == -1
    lib.dlm_free(None)
    # injected host allocation failures, at the first and a later point
    cfg = _cfg(L, shape)
    wb = lib.dlm_weights_bytes(ctypes.byref(cfg))
    for n in (1, 2, 3):
        assert lib.dlm_debug_fail_host_alloc(n) == 0
        got = [lib.dlm_weights_bytes(ctypes.byref(cfg)) for _ in range(n)]
        assert got[:-1] == [wb] * (n - 1) and got[-1] == 0, (n, got)
        assert b"allocation" in lib.dlm_last_error()
    assert lib.dlm_debug_fail_host_alloc(1) == 0
    h = ctypes.c_void_p(1)
    assert lib.dlm_load_synthetic_weights(ctypes.byref(cfg), 0, ctypes.c_void_p(256), 0, None,
                                          ctypes.byref(h)) == -6
    assert h.value is None
    assert lib.dlm_debug_fail_host_alloc(0) == 0
    assert lib.dlm_weights_bytes(ctypes.byref(cfg)) == wb
    # long error messages are copied, not referenced
    for _ in range(100):
        lib.dlm_load_synthetic_weights(ctypes.byref(cfg), 0, ctypes.c_void_p(256), 1, None, ctypes.byref(h))
    assert b"too small" in lib.dlm_last_error()


def oracle(path: str, kat: str) -> None:
    lib = ctypes.CDLL(path)
    lib.oracle_philox4x32_10.argtypes = [ctypes.POINTER(ctypes.c_uint32)] * 3
    lib.oracle_philox4x32_10.restype = None
    lib.oracle_irwin_hall.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint64,
                                      ctypes.c_void_p]
    rows = 0
    with open(kat) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            w = [int(t, 16) for t in line.split()]
            c = (ctypes.c_uint32 * 4)(*w[0:4])
            k = (ctypes.c_uint32 * 2)(*w[4:6])
            o = (ctypes.c_uint32 * 4)()
            lib.oracle_philox4x32_10(c, k, o)
            assert list(o) == w[6:10], (w, list(o))
            rows += 1
    assert rows >= 3
    out = (ctypes.c_int32 * 1000)()
    lib.oracle_irwin_hall(0x1234, 7, 5, 1000, ctypes.cast(out, ctypes.c_void_p))
    assert all(-131070 <= v <= 131070 for v in out)


if __name__ == "__main__":
    assert hasattr(ctypes.CDLL(None), "__asan_init"), "the ASan runtime is not loaded"
    if sys.argv[1] == "abi":
        abi(sys.argv[2])
    else:
        oracle(sys.argv[2], sys.argv[3])
    print("host checks passed", flush=True)
