"""Helpers for GPU parity tests (comparison metrics, GPU availability)."""

from __future__ import annotations

import os
import sys

import numpy as np
import pytest

HIDDEN_TOL = 2e-2      # max-abs-relative error for hidden states and logits
MARGIN = 1e-2          # top-1/top-2 logit margin and |conf - tau| exemption width


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def need_gpu():
    if not gpu_available():
        pytest.skip("no GPU")
    from paper_2608_02625_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        raise RuntimeError("libdlm.so is not built; a GPU test must not pass without the HIP library")


def max_abs_rel(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-30))


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def shape_dict(shape):
    return shape.as_dict()


def decisions_exempt(margin, conf, tau, extra=None):
    """Positions exempt from bit-exact decision checks."""
    ex = (np.asarray(margin) <= MARGIN) | (np.abs(np.asarray(conf) - tau) <= MARGIN)
    if extra is not None:
        ex |= extra
    return ex
