"""Static checks on the generated gfx950 code of the dK/dV kernel.

The D=128 dK/dV kernel keeps its accumulators in AGPRs through inline-asm
MFMAs.  The compiler cannot see the latency of an instruction inside an asm
statement, so two hazards are the kernel's own responsibility:

  * a VALU write of an MFMA's A/B register needs two wait states before the
    MFMA reads it;
  * no other instruction may read or copy an accumulator register before the
    drain (a long run of s_nop with the accumulators tied as operands) that
    follows the last MFMA.

This test compiles the kernel source to device assembly (CPU only) and checks
both in program order, so a compiler change that moves or copies those
registers fails here instead of producing wrong gradients on the GPU.
"""
from __future__ import annotations

import re
import shutil
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
CSRC = ROOT / "paper_2512_22234_amd" / "csrc"
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
KERNEL = "_ZN2bd12_GLOBAL__N_111dkdv_kernelILi128EEEvNS0_9DkvParamsE"


def _regs(tok: str) -> set:
    m = re.fullmatch(r"([va])\[(\d+):(\d+)\]", tok)
    if m:
        return {(m.group(1), r) for r in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.fullmatch(r"([va])(\d+)", tok)
    return {(m.group(1), int(m.group(2)))} if m else set()


def _kernel_instructions(asm: str, name: str):
    lines = asm.split("\n")
    start = next(i for i, l in enumerate(lines) if l.split(";")[0].strip() == name + ":")
    out, in_asm = [], False
    for l in lines[start + 1:]:
        s = l.strip()
        if s.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if s.startswith(";;#ASMEND"):
            in_asm = False
            continue
        if s.startswith(".Lfunc_end"):
            break
        s = s.split(";")[0].strip()
        if not s or s.startswith(".") or s.endswith(":"):
            continue
        parts = s.replace(",", " ").split()
        out.append((parts[0], parts[1:], in_asm))
    return out


def _hazards(insts):
    problems, acc = [], set()
    drain = None
    for k, (op, args, in_asm) in enumerate(insts):
        if in_asm and op.startswith("v_mfma") and args[0].startswith("a"):
            acc |= _regs(args[0])
            srcs = _regs(args[1]) | _regs(args[2])
            waits = 0
            for kk in range(k - 1, -1, -1):  # two wait states back
                if waits >= 2:
                    break
                op2, args2, _ = insts[kk]
                if op2.startswith("v_") and not op2.startswith("v_mfma") and args2 and _regs(args2[0]) & srcs:
                    problems.append(f"VALU write {op2} {args2[0]} feeds an asm MFMA within 2 wait states")
                waits += int(args2[0], 0) + 1 if op2 == "s_nop" else 1
        if in_asm and op == "s_nop" and args[0] == "7":
            drain = k
    assert acc, "no AGPR-pinned MFMAs found"
    assert drain is not None, "no drain found"
    for k, (op, args, in_asm) in enumerate(insts):
        if in_asm or k > drain:
            continue
        touched = set().union(*(_regs(a) for a in args)) if args else set()
        if touched & acc:
            problems.append(f"{op} {' '.join(args)} touches an accumulator before the drain")
    return problems, len(acc)


@pytest.fixture(scope="module")
def dkdv_asm(tmp_path_factory):
    if not Path(HIPCC).exists():
        pytest.skip("hipcc not available")
    from paper_2512_22234_amd.build import compile_flags
    out = tmp_path_factory.mktemp("isa") / "bwd.s"
    flags = [f for f in compile_flags("bwd.hip") if f != "-fPIC"]
    cmd = [HIPCC, *flags, f"-I{CSRC}", "--cuda-device-only", "-S", "-o", str(out), str(CSRC / "bwd.hip")]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    return out.read_text()


def test_dkdv_agpr_accumulators_hazard_free(dkdv_asm):
    problems, n = _hazards(_kernel_instructions(dkdv_asm, KERNEL))
    assert n == 128, n  # 4 dK + 4 dV accumulators of 16 registers
    assert not problems, problems[:10]


def test_checker_flags_early_read():
    """The checker itself: a copy of an accumulator before the drain, and a VALU
    write right before an asm MFMA, are both reported."""
    asm = "\n".join([
        "k:",
        ";;#ASMSTART", "v_mfma_f32_32x32x16_bf16 a[0:15], v[0:3], v[4:7], a[0:15]", ";;#ASMEND",
        "v_accvgpr_read_b32 v20, a3",
        "v_cvt_pk_bf16_f32 v4, v8, v9",
        ";;#ASMSTART", "v_mfma_f32_32x32x16_bf16 a[0:15], v[0:3], v[4:7], a[0:15]", ";;#ASMEND",
        ";;#ASMSTART", "s_nop 7", ";;#ASMEND",
        "v_accvgpr_read_b32 v21, a4",
        "s_endpgm",
        ".Lfunc_end0:",
    ])
    problems, _ = _hazards(_kernel_instructions(asm, "k"))
    assert any("before the drain" in p for p in problems)
    assert any("feeds an asm MFMA" in p for p in problems)
    assert len(problems) == 2
