"""Static checks on the generated gfx950 code (CPU only: hipcc cross-compiles).

The kernels' launch shapes depend on register and LDS budgets that only the
compiler's output shows:

  * the dK/dV kernel runs eight waves per workgroup, two per SIMD, so each
    wave may use at most 256 registers (VGPRs and AGPRs together) or the
    launch fails;
  * the forward and dQ kernels are written for two 256-thread workgroups per
    CU (same limit), and the dK/dV kernel's LDS must fit one CU's 160 KiB;
  * no kernel may spill to scratch memory (a silent, large slowdown).

Each source is compiled to device assembly with the library's own flags and
the kernel metadata is checked, so a change that breaks a budget fails here
instead of at launch time on the GPU.
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
LDS_PER_CU = 160 * 1024


def _metadata(asm: str) -> dict:
    """Kernel name -> {field: int} from the AMDGPU metadata block of a .s file."""
    out = {}
    for block in re.split(r"\n\s+- \.", asm):
        name = re.search(r"\.name:\s+(\S+)", block)
        if not name or not name.group(1).startswith("_Z"):
            continue
        fields = {}
        for key in ("vgpr_count", "agpr_count", "sgpr_count", "private_segment_fixed_size",
                    "group_segment_fixed_size"):
            m = re.search(r"\.?" + key + r":\s+(\d+)", "." + block)
            if m:
                fields[key] = int(m.group(1))
        out[name.group(1)] = fields
    return out


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    if not Path(HIPCC).exists():
        pytest.skip("hipcc not available")
    from paper_2512_22234_amd.build import compile_flags
    meta = {}
    for src in ("fwd.hip", "bwd.hip"):
        out = tmp_path_factory.mktemp("isa") / (src + ".s")
        flags = [f for f in compile_flags(src) if f != "-fPIC"]
        cmd = [HIPCC, *flags, f"-I{CSRC}", "--cuda-device-only", "-S", "-o", str(out), str(CSRC / src)]
        r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
        assert r.returncode == 0, r.stderr[-2000:]
        meta.update(_metadata(out.read_text()))
    return meta


def _find(meta, part):
    found = {k: v for k, v in meta.items() if part in k}
    assert found, f"no kernel matching {part}"
    return found


def test_no_scratch_spills(kernels):
    assert len(kernels) >= 6  # fwd, dkdv, dq at D = 64 and 128
    for name, f in kernels.items():
        assert f.get("private_segment_fixed_size", 0) == 0, name


@pytest.mark.parametrize("part", ["dkdv_kernelILi128", "dkdv_kernelILi64", "fwd_kernelILi128",
                                  "fwd_kernelILi64", "dq_kernelILi128", "dq_kernelILi64"])
def test_two_waves_per_simd_fit(kernels, part):
    for name, f in _find(kernels, part).items():
        # gfx950 metadata: vgpr_count counts architectural VGPRs, agpr_count the
        # accumulation registers; a wave's allocation is their sum (each rounded
        # to 8), and two waves share a SIMD's 512
        total = -(-f["vgpr_count"] // 8) * 8 + -(-f.get("agpr_count", 0) // 8) * 8
        assert total <= 256, (name, f)


def test_dkdv_lds_fits_one_cu(kernels):
    for name, f in _find(kernels, "dkdv_kernel").items():
        assert 0 < f["group_segment_fixed_size"] <= LDS_PER_CU, (name, f)


def test_metadata_parser():
    asm = "\n".join([
        "amdhsa.kernels:",
        "  - .agpr_count:     4",
        "    .group_segment_fixed_size: 1024",
        "    .name:           _Zfoo",
        "    .private_segment_fixed_size: 16",
        "    .sgpr_count:     20",
        "    .vgpr_count:     100",
        "  - .agpr_count:     0",
        "    .name:           _Zbar",
        "    .vgpr_count:     12",
    ])
    m = _metadata(asm)
    assert m["_Zfoo"] == {"vgpr_count": 100, "agpr_count": 4, "sgpr_count": 20,
                          "private_segment_fixed_size": 16, "group_segment_fixed_size": 1024}
    assert m["_Zbar"]["vgpr_count"] == 12 and m["_Zbar"]["agpr_count"] == 0
