"""The four-wave extend kernel issues its P V MFMAs as inline assembly, which the
compiler's hazard recognizer does not see.  This test compiles the kernel source to
gfx950 assembly with the library's own flags and checks the two hazards the kernel
handles by hand:

* a vector instruction (other than a dot product) that writes a register an assembly
  MFMA reads needs two wait states before that MFMA;
* a read of an assembly MFMA's accumulator registers by a non-MFMA instruction needs
  the MFMA's passes plus a few wait states after it (24 are required here).

Wait states are counted as one per instruction and N + 1 for `s_nop N`."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2606_16824_amd import build as b

SRC = os.path.join(b.CSRC, "kernels", "extend_w64.hip")


def _regs(tok):
    out = set()
    for m in re.finditer(r"\b([va])\[(\d+):(\d+)\]|\b([va])(\d+)\b", tok):
        if m.group(1):
            out.update((m.group(1), r) for r in range(int(m.group(2)), int(m.group(3)) + 1))
        else:
            out.add((m.group(4), int(m.group(5))))
    return out


def _instructions(asm: str):
    ins, inasm = [], False
    for line in asm.splitlines():
        s = line.strip()
        if s.startswith(";;#ASMSTART"):
            inasm = True
            continue
        if s.startswith(";;#ASMEND"):
            inasm = False
            continue
        if not s or s.startswith(";") or s.endswith(":") or s.startswith("."):
            continue
        ins.append((s.split(";")[0].strip(), inasm))
    return ins


def _wait_states(s):
    m = re.match(r"s_nop\s+(\d+)", s)
    return int(m.group(1)) + 1 if m else 1


def find_hazards(asm: str):
    ins = _instructions(asm)
    found = []
    for i, (s, in_asm) in enumerate(ins):
        if not (in_asm and s.startswith("v_mfma")):
            continue
        ops = s.split(None, 1)[1].split(",")
        srcs = set().union(*[_regs(o) for o in ops[1:]])
        ws, j = 0, i - 1
        while j >= 0 and ws < 2:
            p = ins[j][0]
            if not p.startswith("s_nop") and p.startswith("v_") and not p.startswith("v_mfma") \
                    and "dot" not in p.split()[0] and len(p.split()) > 1:
                if _regs(p.split(None, 1)[1].split(",")[0]) & srcs:
                    found.append(("vector write before assembly MFMA", p, s))
            ws += _wait_states(p)
            j -= 1
        dst = _regs(ops[0])
        ws, j = 0, i + 1
        while j < len(ins) and ws < 24:
            p, p_asm = ins[j]
            if not (p_asm and p.startswith("v_mfma")) and not p.startswith("s_nop") \
                    and p.split()[0].startswith(("v_", "global_", "buffer_", "ds_")) and len(p.split()) > 1:
                if _regs(p.split(None, 1)[1]) & dst:
                    found.append(("accumulator read after assembly MFMA", s, p))
            ws += _wait_states(p)
            j += 1
    return found


def test_checker_finds_planted_hazards():
    asm = "\n".join([
        "v_cvt_pk_bf16_f32 v4, v1, v2",
        ";;#ASMSTART",
        "v_mfma_f32_32x32x16_bf16 a[0:15], v[4:7], v[8:11], a[0:15]",
        ";;#ASMEND",
        "v_accvgpr_read_b32 v1, a3",
    ])
    kinds = sorted(k for k, _, _ in find_hazards(asm))
    assert kinds == ["accumulator read after assembly MFMA", "vector write before assembly MFMA"]
    safe = "\n".join([
        "v_cvt_pk_bf16_f32 v4, v1, v2",
        "s_nop 1",
        ";;#ASMSTART",
        "v_mfma_f32_32x32x16_bf16 a[0:15], v[4:7], v[8:11], a[0:15]",
        ";;#ASMEND",
        ";;#ASMSTART",
        "s_nop 7\n s_nop 7\n s_nop 7",
        ";;#ASMEND",
        "v_accvgpr_read_b32 v1, a3",
    ])
    assert find_hazards(safe) == []


@pytest.mark.skipif(shutil.which(b.HIPCC) is None and not os.path.exists(b.HIPCC), reason="hipcc missing")
def test_w64_kernel_assembly_has_no_unhandled_hazards(tmp_path):
    out = tmp_path / "w64.s"
    cmd = [b.HIPCC, *b.COMMON, "-x", "hip", "--cuda-device-only", "-S", SRC, "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    asm = out.read_text()
    assert asm.count("v_mfma_f32_32x32x16_bf16 a[") > 0, "no assembly MFMA found"
    hz = find_hazards(asm)
    assert hz == [], hz[:5]
