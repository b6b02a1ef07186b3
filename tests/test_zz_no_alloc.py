"""dlm_refine_step_static (the workspace in the library's static device
array; the call allocates nothing) against dlm_refine_step with a caller
workspace: identical tokens, top-1, confidences and counters, on two calls in
a row with the second on a smaller input, for a dense and a mixture-of-experts
model; a shape whose workspace exceeds the array is refused with nothing
written."""

from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_util import log, need_gpu
from workloads import MODELS
from workloads.inputs import draw_tokens

pytestmark = pytest.mark.gpu


def _inputs(shape, B, P, D, seed):
    rng = np.random.default_rng(seed)
    toks = draw_tokens(rng, (B, P + D), shape.vocab)
    toks[:, P::4] = shape.mask_id                    # some [MASK] slots in the draft
    return toks


def _both(R, toks, P, tau):
    import torch
    B, S = toks.shape
    D = S - P
    out = []
    for static in (False, True):
        g = torch.tensor(toks, device="cuda")
        t1 = torch.full((B * D,), -7, dtype=torch.int32, device="cuda")
        cf = torch.full((B * D,), -7.0, dtype=torch.float32, device="cuda")
        st = torch.full((5,), -7, dtype=torch.int32, device="cuda")
        if static:
            R.refine_step_static(g, P, tau, top1=t1, conf=cf, stats=st)
        else:
            R.refine_step(g, P, tau, top1=t1, conf=cf, stats=st)
        torch.cuda.synchronize()
        out.append((g.cpu().numpy(), t1.cpu().numpy(), cf.cpu().numpy(), st.cpu().numpy()))
    return out


@pytest.mark.parametrize("name,over,calls", [
    ("tiny", dict(lm_head_scale=10.0), [(3, 40, 88, 1), (1, 8, 20, 2)]),
    ("small_moe", dict(lm_head_scale=12.0), [(1, 128, 384, 3), (2, 16, 48, 4)]),
])
def test_static_step_matches_workspace_step(name, over, calls):
    need_gpu()
    import ctypes
    from paper_2608_02625_amd import Refiner
    from paper_2608_02625_amd._lib import STATIC_SCRATCH_BYTES
    shape = MODELS[name].replace(**over)
    R = Refiner(shape.as_dict(), 5)
    for (B, P, D, seed) in calls:                     # the second call is the smaller one
        need = R.lib.dlm_workspace_bytes(ctypes.byref(R.cfg), B, P, D)
        assert 0 < need <= STATIC_SCRATCH_BYTES
        toks = _inputs(shape, B, P, D, seed)
        (ga, ta, ca, sa), (gb, tb, cb, sb) = _both(R, toks, P, 0.3)
        log(f"[static scratch {name}] B={B} P={P} D={D} workspace {need} bytes; stats {sa.tolist()} / {sb.tolist()}")
        assert np.array_equal(ga, gb) and np.array_equal(ta, tb)
        assert np.array_equal(ca.view(np.uint32), cb.view(np.uint32))
        assert np.array_equal(sa, sb) and sa[0] + sa[1] > 0 and sa[4] == 0
        assert np.array_equal(ga[:, :P], toks[:, :P])


def test_static_step_refuses_shapes_beyond_the_array():
    need_gpu()
    import ctypes
    import torch
    from paper_2608_02625_amd import DlmError, Refiner
    from paper_2608_02625_amd._lib import STATIC_SCRATCH_BYTES
    shape = MODELS["tiny"]
    R = Refiner(shape.as_dict(), 5)
    B, P, D = 64, 0, 1024
    assert R.lib.dlm_workspace_bytes(ctypes.byref(R.cfg), B, P, D) > STATIC_SCRATCH_BYTES
    toks = _inputs(shape, B, P, D, 9)
    g = torch.tensor(toks, device="cuda")
    with pytest.raises(DlmError, match="static scratch"):
        R.refine_step_static(g, P, 0.3)
    torch.cuda.synchronize()
    assert np.array_equal(g.cpu().numpy(), toks)
