"""The refinement step captured in a HIP graph and replayed.

A caller may capture `dlm_refine_step` (its own workspace) or
`dlm_refine_step_static` (the library's static scratch) on its stream: every
launch goes to the stream passed, the pass counters are cleared by a kernel
(no memset node), nothing is allocated and nothing synchronises.  Each replay,
from the same starting tokens and with eager library work and
synchronisations between replays, must equal an eager step bit for bit:
tokens, top-1, confidences and counters.
"""

from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_util import log, need_gpu
from workloads import MODELS
from workloads.inputs import draw_tokens

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,over,shape_seed,static", [
    ("tiny", dict(lm_head_scale=10.0), (3, 40, 88, 1), False),
    ("tiny", dict(lm_head_scale=10.0), (3, 40, 88, 1), True),
    ("small_moe", dict(lm_head_scale=12.0), (1, 128, 384, 3), False),
    ("small_moe", dict(lm_head_scale=12.0), (1, 128, 384, 3), True),
])
def test_step_graph_replays_equal_eager_steps(name, over, shape_seed, static):
    need_gpu()
    import torch
    from paper_2608_02625_amd import Refiner
    shape = MODELS[name].replace(**over)
    R = Refiner(shape.as_dict(), 5)
    B, P, D, seed = shape_seed
    tau = 0.3
    rng = np.random.default_rng(seed)
    toks0 = draw_tokens(rng, (B, P + D), shape.vocab).astype(np.int32)
    toks0[:, P::4] = shape.mask_id                   # some [MASK] slots in the draft
    step = R.refine_step_static if static else R.refine_step

    def outputs():
        return (torch.empty(B * D, dtype=torch.int32, device="cuda"),
                torch.empty(B * D, dtype=torch.float32, device="cuda"),
                torch.empty(5, dtype=torch.int32, device="cuda"))

    # eager reference (also the warm-up: workspace, per-kernel caches)
    ref_tok = torch.tensor(toks0, device="cuda")
    r1, rc, rs = outputs()
    step(ref_tok, P, tau, top1=r1, conf=rc, stats=rs)
    torch.cuda.synchronize()
    ref = (ref_tok.cpu().numpy(), r1.cpu().numpy(), rc.cpu().numpy().view(np.uint32), rs.cpu().numpy())
    assert ref[3][0] + ref[3][1] > 0, ref[3]           # the pass edits or unmasks something

    tok = torch.tensor(toks0, device="cuda")
    t1, cf, st = outputs()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                    # warm-up on the capture stream's side
        step(tok, P, tau, top1=t1, conf=cf, stats=st)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(tok, P, tau, top1=t1, conf=cf, stats=st)
    rolled = toks0.copy()
    rolled[:, P:] = np.roll(rolled[:, P:], 1, axis=1)
    other = torch.tensor(rolled, device="cuda")
    for rep in range(3):
        tok.copy_(torch.tensor(toks0, device="cuda"))
        t1.fill_(-7)
        cf.fill_(-7.0)
        st.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        got = (tok.cpu().numpy(), t1.cpu().numpy(), cf.cpu().numpy().view(np.uint32), st.cpu().numpy())
        log(f"[graph {name} static={static}] replay {rep}: stats {got[3].tolist()} (eager {ref[3].tolist()})")
        for a, b in zip(got, ref):
            assert np.array_equal(a, b)
        # eager library work on the same workspace between replays
        step(other, P, tau)
        torch.cuda.synchronize()
