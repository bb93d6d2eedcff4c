"""Static check of the generated gfx950 code: no MFMA inside a lane-masked
region that lacks an execz skip branch.

MFMA instructions do not honour the EXEC mask.  When the compiler cannot prove
a branch condition wave-uniform it predicates the branch body with EXEC and may
drop the skip branch for short bodies; an MFMA there still executes (and
accumulates) when every lane is masked off.  Wave-uniform conditions built from
scalar values (wave_id()) avoid this; the check keeps it that way."""
import os
import re
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_2607_02980_amd import build as B

HIP_SOURCES = [s for s in B.SOURCES if s.endswith(".hip")]


def masked_mfma_regions(asm_lines):
    bad = []
    fn = None
    for i, line in enumerate(asm_lines):
        m = re.match(r"^(_Z\w+):", line)
        if m:
            fn = m.group(1)
        if not ("s_and_saveexec_b64" in line or "s_andn2_saveexec_b64" in line):
            continue
        j = i + 1
        while j < len(asm_lines) and (asm_lines[j].strip().startswith(";") or not asm_lines[j].strip()
                                      or asm_lines[j].startswith(".LBB")):
            j += 1
        guarded = j < len(asm_lines) and "s_cbranch_execz" in asm_lines[j]
        k = j
        has_mfma = False
        while k < len(asm_lines) and not re.search(r"s_or_b64 exec|s_mov_b64 exec|s_endpgm|s_cbranch|s_branch",
                                                   asm_lines[k]):
            has_mfma |= "v_mfma" in asm_lines[k]
            k += 1
        if has_mfma and not guarded:
            bad.append((fn, i + 1))
    return bad


def _asm(src, tmp_path):
    out = os.path.join(tmp_path, src + ".s")
    cmd = [B.HIPCC, *B.FLAGS, "-x", "hip", "--cuda-device-only", "-S", os.path.join(B.CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return open(out).read().splitlines()


@pytest.mark.skipif(not os.path.exists(B.HIPCC), reason="hipcc not available")
def test_no_mfma_under_unguarded_exec_mask(tmp_path):
    with ThreadPoolExecutor(max_workers=len(HIP_SOURCES)) as ex:
        asms = list(ex.map(lambda s: _asm(s, str(tmp_path)), HIP_SOURCES))
    problems = {src: masked_mfma_regions(a)[:5] for src, a in zip(HIP_SOURCES, asms)}
    problems = {k: v for k, v in problems.items() if v}
    assert not problems, problems


def test_checker_flags_a_masked_mfma():
    asm = [
        "_Zkernel:",
        "\tv_cmp_gt_u32_e32 vcc, 32, v1",
        "\ts_and_saveexec_b64 s[0:1], vcc",
        "; %bb.1:",
        "\tv_mfma_f32_16x16x32_bf16 a[0:3], v[2:5], v[6:9], a[0:3]",
        "\ts_or_b64 exec, exec, s[0:1]",
        "\ts_and_saveexec_b64 s[0:1], vcc",
        "\ts_cbranch_execz .LBB0_2",
        "\tv_mfma_f32_16x16x32_bf16 a[0:3], v[2:5], v[6:9], a[0:3]",
        ".LBB0_2:",
        "\ts_or_b64 exec, exec, s[0:1]",
    ]
    assert masked_mfma_regions(asm) == [("_Zkernel", 3)]
