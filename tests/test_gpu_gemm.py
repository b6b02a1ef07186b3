"""The library's bf16 MFMA GEMM on its own against a float32 PyTorch reference
(exact bf16 operands, so the only difference is fp32 summation order)."""

from __future__ import annotations

import pytest

from tests.gpu_util import log, need_gpu

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("m,n,k,tile", [
    (256, 256, 64, (256, 256)),
    (300, 200, 128, (256, 256)),      # ragged in m and n
    (1000, 520, 512, (256, 128)),
    (77, 600, 192, (128, 256)),
    (513, 129, 256, (128, 128)),
    (130, 70, 64, (128, 64)),
    (1, 1, 64, (128, 64)),
    # 8-wave 256x256 tiles: 2+2 stages, a third B stage, a third A stage
    (600, 520, 640, ((2 << 16) | 256, 256)),
    (600, 520, 640, ((5 << 16) | 256, 256)),
    (777, 300, 1088, ((6 << 16) | 256, 256)),
    (256, 256, 64, ((5 << 16) | 256, 256)),
    # ping-pong schedule (2 + 3 and 3 + 2 stages): one K tile, short K with a
    # prologue per tile, continuous copies, and more tiles than resident
    # workgroups (several output tiles per workgroup) with short and long K
    (256, 256, 64, ((11 << 16) | 256, 256)),
    (300, 200, 128, ((11 << 16) | 256, 256)),
    (600, 520, 640, ((11 << 16) | 256, 256)),
    (777, 300, 1088, ((12 << 16) | 256, 256)),
    (1, 1, 64, ((12 << 16) | 256, 256)),
    (8229, 2100, 128, ((11 << 16) | 256, 256)),
    (8229, 2100, 320, ((11 << 16) | 256, 256)),
    (8229, 2100, 320, ((12 << 16) | 256, 256)),
])
def test_gemm_matches_fp32_reference(m, n, k, tile):
    need_gpu()
    import torch
    from paper_2608_02625_amd.model import debug_gemm
    g = torch.Generator(device="cpu").manual_seed(m * 131 + n * 7 + k)
    a = torch.randn(m, k, generator=g).to(torch.bfloat16).cuda()
    b = torch.randn(n, k, generator=g).to(torch.bfloat16).cuda()
    c = debug_gemm(a, b, tile)
    ref = a.float().cpu() @ b.float().cpu().T
    err = ((c.cpu() - ref).abs().max() / ref.abs().max()).item()
    log(f"[gemm {m}x{n}x{k} tile {tile}] max-abs-rel {err:.2e}")
    assert err < 1e-5
