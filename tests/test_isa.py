"""Static checks on the gfx950 assembly of the library's kernels (produced
by the build next to the objects; no GPU needed).

An MFMA issued inside a region where EXEC was narrowed by a divergent branch
still updates its accumulators for every lane, so such a region must be
skipped with s_cbranch_execz when EXEC is empty; the kernels keep all MFMA
control flow wave-uniform so that this never arises."""

from __future__ import annotations

import glob
import os
import re

import pytest

BUILD = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2608_02625_amd", "_build")


def _functions(path):
    text = open(path).read()
    for m in re.finditer(r"^(_Z\S+):\s*;", text, re.M):
        end = text.index(".Lfunc_end", m.end())
        lines = [l.strip() for l in text[m.end():end].splitlines()]
        yield m.group(1), [l for l in lines if l and not l.startswith(";")]


def masked_mfmas(lines):
    """MFMAs issued after an EXEC-narrowing s_and_saveexec that is not
    followed by a branch on EXEC being empty (s_cbranch_execz over the region,
    or s_cbranch_execnz into a region placed out of line), before EXEC is
    restored."""
    bad, masked = 0, False
    for i, l in enumerate(lines):
        op = l.split()[0]
        if "saveexec" in op:
            nxt = lines[i + 1].split()[0] if i + 1 < len(lines) else ""
            masked = nxt not in ("s_cbranch_execz", "s_cbranch_execnz")
        elif op.startswith("s_or_b64") and "exec, exec" in l:
            masked = False
        elif op.startswith("v_mfma") and masked:
            bad += 1
    return bad


def test_scanner_flags_a_masked_mfma():
    lines = ["v_cmp_lt_i32_e64 s[4:5], v11, v3", "s_and_saveexec_b64 s[8:9], s[4:5]",
             "v_mfma_f32_32x32x16_bf16 a[0:15], v[44:47], v[72:75], a[0:15]", "s_or_b64 exec, exec, s[8:9]"]
    assert masked_mfmas(lines) == 1
    lines.insert(2, "s_cbranch_execz .LBB0_3")
    assert masked_mfmas(lines) == 0
    lines[2] = "s_cbranch_execnz .LBB0_3"
    assert masked_mfmas(lines) == 0


def test_no_mfma_under_exec_mask():
    files = sorted(glob.glob(os.path.join(BUILD, "*.s")))
    if not files:
        pytest.skip("library assembly not built (run the build first)")
    offenders = []
    n_mfma_kernels = 0
    for f in files:
        for name, lines in _functions(f):
            if any(l.startswith("v_mfma") for l in lines):
                n_mfma_kernels += 1
            bad = masked_mfmas(lines)
            if bad:
                offenders.append((os.path.basename(f), name, bad))
    assert n_mfma_kernels > 0
    assert not offenders, offenders
