"""Machine-code checks of the bf16 attention kernels, compiled here for gfx950.

The MLA kernel keeps its output accumulators in the AGPR file and updates them
only with MFMAs written as inline assembly; the compiler schedules around
those statements without knowing that they are MFMAs.  A result of such an
MFMA is readable 18 wait states after it issues.  These tests compile the
kernels exactly as the build does and walk the generated assembly:

  * no instruction other than an MFMA reads or writes a register that an
    inline-assembly MFMA wrote until an s_nop sequence of at least 18 wait
    states has passed (the kernels' explicit wait before the epilogue);
  * no accumulator is copied between AGPRs (v_accvgpr_mov), which the
    compiler only does when it moves a value it does not see being written.

The walker is checked on a small synthetic listing first."""
import os
import re
import subprocess

import pytest

from paper_2606_17107_amd import build as B

pytestmark = pytest.mark.skipif(not os.path.exists(B.hipcc()), reason="hipcc not available")


def _regs(tok):
    m = re.match(r"^([va])(\d+)$", tok)
    if m:
        return {(m.group(1), int(m.group(2)))}
    m = re.match(r"^([va])\[(\d+):(\d+)\]$", tok)
    if m:
        return {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    return set()


def _split(line):
    body = line.split(";")[0].strip()
    parts = body.split(None, 1)
    if not parts:
        return "", []
    if len(parts) == 1:
        return parts[0], []
    return parts[0], [o.strip() for o in re.split(r",(?![^\[]*\])", parts[1])]


def hazards(asm_text):
    """(kernel, line, kind, text) for every violation in an assembly listing."""
    found = []
    starts = [m.start() for m in re.finditer(r"^_ZN\S*kernel\S*:", asm_text, re.M)]
    for s0 in starts:
        name = asm_text[s0:asm_text.index(":", s0)]
        end = asm_text.find(".Lfunc_end", s0)
        lines = asm_text[s0:end if end > 0 else len(asm_text)].split("\n")
        pending, nops, in_asm = set(), 0, False
        for k, line in enumerate(lines):
            if ";;#ASMSTART" in line:
                in_asm = True
                continue
            if ";;#ASMEND" in line:
                in_asm = False
                continue
            op, ops = _split(line)
            if not op or op.endswith(":") or op.startswith(".") or op.startswith(";"):
                continue
            if op == "v_accvgpr_mov_b32":
                found.append((name, k, "AGPR copy", line.strip()))
            if op == "s_nop":
                nops += int(ops[0], 0) + 1
                if nops >= 18:
                    pending.clear()
                continue
            nops = 0
            if op.startswith("v_mfma"):
                srcs = set().union(*(_regs(o) for o in ops[1:3]))
                if srcs & pending:
                    found.append((name, k, "MFMA operand read before the wait", line.strip()))
                if in_asm:
                    pending |= _regs(ops[0])
                else:
                    pending -= _regs(ops[0])
                continue
            regs = set().union(*(_regs(o) for o in ops)) if ops else set()
            if regs & pending:
                found.append((name, k, "result used before the wait", line.strip()))
    return found


def test_walker_flags_early_reads():
    ok = """_ZN3fooL6kernelEv:
	;;#ASMSTART
	v_mfma_f32_32x32x16_bf16 a[0:15], v[0:3], v[4:7], a[0:15]
	;;#ASMEND
	v_add_f32_e32 v8, v9, v10
	;;#ASMSTART
	s_nop 7
	s_nop 7
	s_nop 7
	;;#ASMEND
	v_accvgpr_read_b32 v11, a3
.Lfunc_end0:
"""
    assert hazards(ok) == []
    early = ok.replace("	v_add_f32_e32 v8, v9, v10\n", "	v_accvgpr_read_b32 v8, a2\n")
    assert [h[2] for h in hazards(early)] == ["result used before the wait"]
    copy = ok.replace("	v_add_f32_e32 v8, v9, v10\n", "	v_accvgpr_mov_b32 a40, a2\n")
    assert {h[2] for h in hazards(copy)} == {"AGPR copy", "result used before the wait"}
    # the compiler's own MFMAs are left to the compiler
    builtin = ok.replace(";;#ASMSTART\n	v_mfma", ";\n	v_mfma", 1)
    assert hazards(builtin.replace("	v_add_f32_e32 v8, v9, v10\n", "	v_accvgpr_read_b32 v8, a2\n")) == []


@pytest.mark.parametrize("src", ["attn_mla_bf16.hip", "attn_gqa_bf16.hip"])
def test_attention_kernel_assembly(src, tmp_path):
    path = os.path.join(B.CSRC, src)
    out = tmp_path / (src + ".s")
    cmd = [B.hipcc()] + B.compile_flags() + B.FILE_FLAGS.get(src, []) + [
        "--cuda-device-only", "-S", path, "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    text = out.read_text()
    assert "v_mfma" in text
    found = hazards(text)
    assert not found, found[:10]
