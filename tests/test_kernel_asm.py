"""Static checks of the gfx950 assembly hipcc generates for the kernels (no GPU needed).

* The fused kernel's P V MFMAs are written as inline assembly (accumulating into AGPRs in the
  long instance, into VGPRs in the short one), so the compiler's hazard recognizer does not pad them:
  where the kernel omits the wait states in front of such an MFMA it relies on no VALU instruction
  having written one of its source registers just before. gfx950 needs two wait
  states between a VALU write of a VGPR and an MFMA that reads it; this is checked in the code.
* Some loads into registers are inline assembly the compiler does not track (Q in the fused kernel,
  P in the layer-by-layer P V kernel): the kernels order them with explicit vmcnt waits. The check
  follows every path of each kernel, keeps the queue of vector-memory operations in issue order
  (vmcnt retires the oldest first) and fails if any instruction touches a register of a load that
  may still be in flight.
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


def _asm(source):
    d = tempfile.mkdtemp(prefix="fa_asm_")
    try:
        out = os.path.join(d, "kernel.s")
        fa_build.kernel_asm(out, source)
        return open(out).read()
    finally:
        shutil.rmtree(d, ignore_errors=True)


@pytest.fixture(scope="module")
def asm_text():
    return _asm("fa_fwd_kernel.hip")


@pytest.fixture(scope="module")
def lbl_asm_text():
    return _asm("fa_lbl_kernel.hip")


@pytest.fixture(scope="module")
def decode_asm_text():
    return _asm("fa_decode_kernel.hip")


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
        if not s or (s.startswith(".") and not s.endswith(":")):
            continue  # directives; local labels (".LBB0_1:") are kept
        out.append(("label", s) if s.endswith(":") else ("ins", s))
    return out


def test_no_packed_fp32_valu(asm_text):
    hits = re.findall(r"\bv_pk_(?:add|mul|fma)_f32\b", asm_text)
    assert not hits, f"{len(hits)} packed fp32 VALU instructions in the kernel"


def test_no_scratch(asm_text):
    sizes = re.findall(r"\.amdhsa_private_segment_fixed_size\s+(\d+)", asm_text)
    assert sizes, "no kernel descriptor found"
    assert all(int(x) == 0 for x in sizes), f"kernels use scratch memory: {sizes}"


# ---------------------------------------------------------------------------------------------
# registers of in-flight loads
# ---------------------------------------------------------------------------------------------

_VMEM = re.compile(r"^(buffer|global|flat)_(load|store|atomic)")


def _kernels(text):
    """{kernel name: [(kind, text, from_inline_asm)]} for every kernel in the assembly, from its entry
    label to its .Lfunc_end label; kind is "label" or "ins"."""
    out, cur, in_asm = {}, None, False
    for line in text.split("\n"):
        if ";;#ASMSTART" in line:
            in_asm = True
        elif ";;#ASMEND" in line:
            in_asm = False
        s = line.split(";")[0].strip()
        if not s or (s.startswith(".") and not s.endswith(":")):
            continue
        if s.endswith(":"):
            if re.fullmatch(r"_Z\w+:", s):
                cur = out.setdefault(s[:-1], [])
                continue
            if s.startswith(".Lfunc_end"):
                cur = None
                continue
            if cur is not None:
                cur.append(("label", s, False))
        elif cur is not None:
            cur.append(("ins", s, in_asm))
    return out


def _operands(s):
    parts = s.split(None, 1)
    return [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []


def _in_flight_violations(code):
    """Flow every reachable (instruction, in-flight queue) state through the kernel's branches;
    return the instructions that touch a register of an inline-asm load that may still be in
    flight (the compiler orders its own loads itself; its waits only count those, and untracked
    operations can only make them stricter). The queue holds every outstanding vector-memory
    operation in issue order, with the destination registers of inline-asm loads (empty for the
    rest); vmcnt(N) keeps the newest N. The hardware counter holds at most 63 operations, so older
    entries are retired, which bounds the states."""
    labels = {s[:-1]: i for i, (k, s, _) in enumerate(code) if k == "label"}
    problems, seen = set(), set()
    work = [(0, ())]
    while work:
        i, queue = work.pop()
        while i < len(code):
            if (i, queue) in seen:
                break
            seen.add((i, queue))
            kind, s, from_asm = code[i]
            if kind == "label":
                i += 1
                continue
            op = s.split()[0]
            ops = _operands(s)
            if op == "s_endpgm":
                break
            if op == "s_waitcnt":
                m = re.search(r"vmcnt\((\d+)\)", s)
                if m:
                    n = int(m.group(1))
                    queue = queue[len(queue) - n:] if n < len(queue) else queue
                i += 1
                continue
            busy = frozenset().union(*queue)
            if _VMEM.match(op):
                is_load = "_load" in op and not s.endswith(" lds")
                dst = _regs(ops[0]) if is_load else set()
                srcs = set().union(*(_regs(o) for o in (ops[1:] if is_load else ops)))
                if (dst | srcs) & busy:
                    problems.add(s)
                queue = (queue + (frozenset(dst) if from_asm else frozenset(),))[-63:]
            elif ops and set().union(*(_regs(o) for o in ops)) & busy:
                problems.add(s)
            if op.startswith("s_cbranch") or op == "s_branch":
                tgt = labels.get(ops[0])
                assert tgt is not None, f"branch to unknown label: {s}"
                if op == "s_branch":
                    i = tgt
                    continue
                work.append((tgt, queue))
            i += 1
    return sorted(problems)


def test_inline_asm_mfma_operands_settled(asm_text):
    """Every inline-asm MFMA (the P V product, accumulating into AGPRs in the long instance and into
    VGPRs in the short one) has no VALU write of one of its source registers within the two wait
    states before it (the compiler pads only the MFMAs it emits itself)."""
    checked, forms, problems = 0, set(), []
    for name, code in _kernels(asm_text).items():
        for i, (kind, s, from_asm) in enumerate(code):
            if kind != "ins" or not from_asm or not s.startswith("v_mfma"):
                continue
            checked += 1
            ops = _operands(s)
            forms.add(ops[0][0])
            srcs = _regs(ops[1]) | _regs(ops[2]) | _regs(ops[3])
            ws, j = 0, i - 1
            while j >= 0 and ws < WAIT_STATES:
                k, t, _ = code[j]
                if k == "label":
                    problems.append(f"{name}: branch target within {WAIT_STATES} wait states of: {s}")
                    break
                if t.startswith("s_nop"):
                    ws += int(t.split()[1]) + 1
                else:
                    op = t.split()[0]
                    if op.startswith("v_") and not op.startswith("v_mfma") and " " in t:
                        dst = t.split(None, 1)[1].split(",")[0].strip()
                        if _regs(dst) & srcs:
                            problems.append(f"{name}: {t}  ->  {s}")
                    ws += 1
                j -= 1
    assert checked > 0, "no inline-asm MFMA found in the kernel assembly"
    assert forms == {"a", "v"}, f"expected inline-asm MFMAs into AGPRs and into VGPRs, found {forms}"
    assert not problems, "\n".join(problems[:20])


@pytest.mark.parametrize("which", ["fused", "lbl"])
def test_no_access_to_registers_of_in_flight_loads(which, asm_text, lbl_asm_text):
    kernels = _kernels(asm_text if which == "fused" else lbl_asm_text)
    assert kernels, "no kernel found in the assembly"
    report = {}
    n_asm_loads = 0
    for name, code in kernels.items():
        n_asm_loads += sum(1 for k, t, a in code if a and k == "ins" and re.match(r"(buffer|global)_load", t))
        bad = _in_flight_violations(code)
        if bad:
            report[name] = bad[:5]
    assert n_asm_loads > 0, "no inline-asm load found: the check would be vacuous"
    assert not report, "\n".join(f"{k}: {v}" for k, v in report.items())


@pytest.mark.parametrize("which", ["lbl", "decode"])
def test_other_kernels_no_packed_fp32_no_scratch(which, lbl_asm_text, decode_asm_text):
    text = lbl_asm_text if which == "lbl" else decode_asm_text
    assert not re.findall(r"\bv_pk_(?:add|mul|fma)_f32\b", text)
    sizes = re.findall(r"\.amdhsa_private_segment_fixed_size\s+(\d+)", text)
    assert sizes and all(int(x) == 0 for x in sizes), sizes


def test_decode_no_access_to_registers_of_in_flight_loads(decode_asm_text):
    kernels = _kernels(decode_asm_text)
    assert kernels
    report = {n: bad[:5] for n, code in kernels.items() if (bad := _in_flight_violations(code))}
    assert not report, report


def test_no_scalar_memory_writes(asm_text, lbl_asm_text, decode_asm_text):
    # Every store and atomic goes through the vector memory path.
    for text in (asm_text, lbl_asm_text, decode_asm_text):
        assert not re.findall(r"\bs_(?:store|atomic|buffer_store|dcache_wb|dcache_discard)\w*", text)


def test_buffer_descriptors_in_scalar_registers(asm_text, lbl_asm_text, decode_asm_text):
    # A buffer instruction takes its resource descriptor from four SGPRs. The direct-to-LDS loads are
    # inline assembly with a scalar-register constraint; should a descriptor value ever be computed in
    # vector registers, the compiler substitutes the VGPRs into the instruction text instead of
    # failing, and the load would address through an undefined descriptor.
    for text in (asm_text, lbl_asm_text, decode_asm_text):
        loads = re.findall(r"^\s*(buffer_\w+\s+[^\n]*)$", text, re.M)
        assert loads
        # operands: [vdata,] vaddr, srsrc, soffset: the descriptor is the operand before the last
        bad = [ln for ln in loads if not re.search(r",\s*s\[\d+:\d+\],\s*[^,]+$", ln)]
        assert not bad, bad[:5]
