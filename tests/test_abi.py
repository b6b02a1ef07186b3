"""CPU checks of the C ABI: the library loads, exports every declared entry point,
and its host-side validation and size queries behave (no GPU work is launched)."""

from __future__ import annotations

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dlm.h")


def _lib():
    from paper_2608_02625_amd import _lib as L
    if not os.path.exists(L.LIB_PATH):
        import paper_2608_02625_amd.build as b
        b.build()
    return L


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dlm_[a-z_]+)\s*\(", src)))


def test_header_declares_the_entry_points():
    names = _declared()
    for n in ("dlm_load_synthetic_weights", "dlm_refine_step", "dlm_refine", "dlm_weights_bytes",
              "dlm_workspace_bytes", "dlm_free", "dlm_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    L = _lib()
    lib = ctypes.CDLL(L.LIB_PATH)
    for n in _declared():
        assert hasattr(lib, n), n
    bound = {n for n, _, _ in L.SIGNATURES}
    assert bound == set(_declared())


def _cfg(L, **over):
    from workloads import MODELS
    from paper_2608_02625_amd.model import make_config
    d = MODELS["mini_moe"].as_dict()
    d.update(over)
    return make_config(d)


def test_size_queries_and_validation():
    L = _lib()
    lib = L.load()
    cfg = _cfg(L)
    wb = lib.dlm_weights_bytes(ctypes.byref(cfg))
    # 20 layers of d 2048: QKV 3072x2048, O 2048x2048, router 64x2048, 65 experts of
    # 3 x 1024x2048, plus embedding and LM head 157184x2048, all bf16 (+ gains, padding).
    params = 20 * (3072 * 2048 + 2048 * 2048 + 64 * 2048 + 65 * 3 * 1024 * 2048) + 2 * 157184 * 2048
    assert params * 2 <= wb <= params * 2 + 20 * 16 * 4096 + 4 * 4096 + 200 * 256 * 20
    ws = lib.dlm_workspace_bytes(ctypes.byref(cfg), 8, 256, 384)
    assert ws > 5120 * 2048 * 4
    assert lib.dlm_workspace_bytes(ctypes.byref(cfg), 0, 256, 384) == 0
    assert lib.dlm_workspace_bytes(ctypes.byref(cfg), 8, 256, 0) == 0
    # drafting: the per-layer K and V^T caches of all 640 positions come on top
    # of the window buffers (20 layers x 8 x 4 kv heads x 640 x 128 x 2 bytes each)
    cfg_kv = dict(zip([f for f, _ in L.DlmConfig._fields_], [getattr(cfg, f) for f, _ in L.DlmConfig._fields_]))
    dw = lib.dlm_draft_workspace_bytes(ctypes.byref(cfg), 8, 256, 384, 64)
    cache = 2 * cfg_kv["n_layers"] * 8 * cfg_kv["n_kv_heads"] * 640 * cfg_kv["head_dim"] * 2
    assert dw >= cache + lib.dlm_workspace_bytes(ctypes.byref(cfg), 8, 0, 256)
    assert lib.dlm_draft_workspace_bytes(ctypes.byref(cfg), 8, 256, 384, 0) == 0
    assert lib.dlm_draft_workspace_bytes(ctypes.byref(cfg), 8, 256, 384, 1025) == 0
    for bad in (dict(head_dim=96), dict(top_k=9), dict(mask_id=157184), dict(n_heads=15),
                dict(expert_ffn_dim=100), dict(n_experts=300), dict(vocab=1)):
        assert lib.dlm_weights_bytes(ctypes.byref(_cfg(L, **bad))) == 0, bad
    # Activations are addressed with 32-bit buffer offsets: a [tokens][d_model]
    # bf16 buffer must stay below 2 GiB.  d 2048: 2^19 tokens are 2 GiB exactly.
    assert lib.dlm_workspace_bytes(ctypes.byref(cfg), 512, 0, 1023) > 0        # 523776 tokens
    assert lib.dlm_workspace_bytes(ctypes.byref(cfg), 512, 1, 1023) == 0       # 2^19 tokens
    assert lib.dlm_draft_workspace_bytes(ctypes.byref(cfg), 512, 1, 1023, 64) == 0


def test_errors_are_reported_without_gpu_work():
    L = _lib()
    lib = L.load()
    h = ctypes.c_void_p()
    bad = _cfg(L, head_dim=96)
    st = lib.dlm_load_synthetic_weights(ctypes.byref(bad), 0, None, 0, None, ctypes.byref(h))
    assert st == -1 and b"head_dim" in lib.dlm_last_error()
    good = _cfg(L)
    st = lib.dlm_load_synthetic_weights(ctypes.byref(good), 0, None, 0, None, ctypes.byref(h))
    assert st == -1 and b"NULL" in lib.dlm_last_error()
    st = lib.dlm_load_synthetic_weights(ctypes.byref(good), 0, ctypes.c_void_p(256), 1024, None, ctypes.byref(h))
    assert st == -5 and b"too small" in lib.dlm_last_error()
    assert lib.dlm_refine_step(None, 1, 1, 1, None, 0.5, None, 0, None, None, None, None) == -1
    assert lib.dlm_refine(None, 1, 1, 1, None, None, None, 1, 0.5, None, 0, None, None) == -1
    assert lib.dlm_draft(None, 1, 1, 64, None, None, 64, 16, 0.25, None, 0, None, None, None) == -1
    assert lib.dlm_draft_step(None, 1, 1, 64, 64, 0, 16, 0.25, None, None, 0, None, None, None, None, None) == -1
    with pytest.raises(L.DlmError):
        L.check(-1, "x")


def test_host_allocation_failure_is_a_status():
    """A failed host allocation inside the library (injected at its allocation
    points) comes back as DLM_ERR_NO_MEMORY, leaves no half-built model behind,
    and the next call works: no C++ exception crosses the C ABI."""
    L = _lib()
    lib = L.load()
    cfg = _cfg(L)
    wb = lib.dlm_weights_bytes(ctypes.byref(cfg))
    assert wb > 0
    try:
        assert lib.dlm_debug_fail_host_alloc(1) == 0
        assert lib.dlm_weights_bytes(ctypes.byref(cfg)) == 0
        assert b"allocation" in lib.dlm_last_error()
        assert lib.dlm_weights_bytes(ctypes.byref(cfg)) == wb            # the hook fired once
        # The weight plan is built before any GPU work; with the hook off the
        # same call stops at the size check (weights_bytes 0), so no GPU work
        # is launched either way.
        h = ctypes.c_void_p(1)
        assert lib.dlm_debug_fail_host_alloc(1) == 0
        st = lib.dlm_load_synthetic_weights(ctypes.byref(cfg), 0, ctypes.c_void_p(256), 0, None, ctypes.byref(h))
        assert st == -6 and h.value is None, (st, h.value)
        assert L.STATUS_NAMES[st] == "DLM_ERR_NO_MEMORY"
        st = lib.dlm_load_synthetic_weights(ctypes.byref(cfg), 0, ctypes.c_void_p(256), 0, None, ctypes.byref(h))
        assert st == -5
        # a later allocation point: the second pass through one fails
        assert lib.dlm_debug_fail_host_alloc(2) == 0
        assert lib.dlm_weights_bytes(ctypes.byref(cfg)) == wb
        assert lib.dlm_weights_bytes(ctypes.byref(cfg)) == 0
        assert lib.dlm_debug_fail_host_alloc(-1) == -1
    finally:
        lib.dlm_debug_fail_host_alloc(0)


def test_bench_refuses_more_than_one_gpu():
    """bench.py runs on one GPU: --gpus 2 exits with status 2 and says why,
    before any GPU work."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""
