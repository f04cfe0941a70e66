"""Static checks of the gfx950 assembly hipcc generates for the attention kernel (no GPU needed).

The P V MFMAs are written as inline assembly, so the compiler's hazard recognizer does not pad them:
where the kernel omits the wait states in front of such an MFMA it relies on no VALU instruction
having written one of its source registers just before. gfx950 needs two wait states between a
VALU write of a VGPR and an MFMA that reads it; this test checks that in the generated code.
"""

import os
import re
import shutil
import tempfile

import pytest

from paper_2609_21264_amd import build as fa_build

WAIT_STATES = 2  # VALU write of a VGPR -> MFMA read of it as SrcA/B/C


def _have_hipcc():
    try:
        fa_build.hipcc()
        return True
    except RuntimeError:
        return False


pytestmark = pytest.mark.skipif(not _have_hipcc(), reason="hipcc not installed")


@pytest.fixture(scope="module")
def asm_text():
    d = tempfile.mkdtemp(prefix="fa_asm_")
    try:
        out = os.path.join(d, "kernel.s")
        fa_build.kernel_asm(out)
        return open(out).read()
    finally:
        shutil.rmtree(d, ignore_errors=True)


def _regs(tok):
    m = re.fullmatch(r"([va])\[(\d+):(\d+)\]", tok)
    if m:
        return {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.fullmatch(r"([va])(\d+)", tok)
    if m:
        return {(m.group(1), int(m.group(2)))}
    return set()


def _instructions(text):
    out = []
    for line in text.split("\n"):
        s = line.split(";")[0].strip()
        if not s or s.startswith("."):
            continue
        out.append(("label", s) if s.endswith(":") else ("ins", s))
    return out


def test_agpr_mfma_operands_settled(asm_text):
    ins = _instructions(asm_text)
    checked, problems = 0, []
    for i, (kind, s) in enumerate(ins):
        if kind != "ins" or not s.startswith("v_mfma"):
            continue
        ops = [o.strip() for o in s.split(None, 1)[1].split(",")]
        if not ops[0].startswith("a"):
            continue  # VGPR-form MFMAs are emitted (and padded) by the compiler itself
        checked += 1
        srcs = _regs(ops[1]) | _regs(ops[2]) | _regs(ops[3])
        ws, j = 0, i - 1
        while j >= 0 and ws < WAIT_STATES:
            k, t = ins[j]
            if k == "label":
                problems.append(f"branch target within {WAIT_STATES} wait states of: {s}")
                break
            if t.startswith("s_nop"):
                ws += int(t.split()[1]) + 1
            else:
                op = t.split()[0]
                if op.startswith("v_") and not op.startswith("v_mfma") and " " in t:
                    dst = t.split(None, 1)[1].split(",")[0].strip()
                    if _regs(dst) & srcs:
                        problems.append(f"{t}  ->  {s}")
                ws += 1
            j -= 1
    assert checked > 0, "no AGPR-accumulator MFMA found in the kernel assembly"
    assert not problems, "\n".join(problems[:20])


def test_no_packed_fp32_valu(asm_text):
    hits = re.findall(r"\bv_pk_(?:add|mul|fma)_f32\b", asm_text)
    assert not hits, f"{len(hits)} packed fp32 VALU instructions in the kernel"


def test_no_scratch(asm_text):
    sizes = re.findall(r"\.amdhsa_private_segment_fixed_size\s+(\d+)", asm_text)
    assert sizes, "no kernel descriptor found"
    assert all(int(x) == 0 for x in sizes), f"kernels use scratch memory: {sizes}"
