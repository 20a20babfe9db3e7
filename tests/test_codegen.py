"""Checks of the generated gfx950 code that the compiler itself cannot make.

The direct-to-LDS GEMM path issues its loads as inline assembly that sets
M0 (the LDS base of a wave's 1 KB) and relies on no compiler-generated code
of those kernels keeping a value in M0; its LDS reads are ordered after the
loads by explicit waits and barriers, so every such load must come from that
assembly.  Compiling the GEMM source to assembly (on the CPU, about half a minute)
checks both for every GEMM kernel instance.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_19528_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


@pytest.fixture(scope="module")
def gemm_asm(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("asm") / "gemm.s"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "--cuda-device-only", "-S",
           os.path.join(CSRC, "gemm.hip"), "-o", str(out)]
    p = subprocess.run(cmd, capture_output=True, text=True)
    assert p.returncode == 0, p.stderr[-2000:]
    return out.read_text()


def _kernels(asm):
    names = re.findall(r"^(_ZN4lora11gemm_kernel[^:\s]+): ;", asm, re.M)
    assert names
    for n in names:
        body = asm[asm.index(n + ": ;"):]
        yield n, body[:body.index(".Lfunc_end")]


def test_m0_only_written_by_the_load_assembly(gemm_asm):
    for name, body in _kernels(gemm_asm):
        outside = re.sub(r";;#ASMSTART.*?;;#ASMEND", "", body, flags=re.S)
        assert not re.search(r"\bm0\b", outside), name


def test_direct_to_lds_loads_come_from_the_assembly(gemm_asm):
    n_dma = 0
    for name, body in _kernels(gemm_asm):
        outside = re.sub(r";;#ASMSTART.*?;;#ASMEND", "", body, flags=re.S)
        assert not re.search(r"buffer_load_dword\S*\s.*\blds\b", outside), name
        inside = re.findall(r";;#ASMSTART(.*?);;#ASMEND", body, flags=re.S)
        for blk in inside:
            if " lds" in blk:
                n_dma += 1
                # wait states: before the load may read SGPRs a vector op wrote, and
                # between the write of M0 and the load
                lines = [l.strip() for l in blk.strip().splitlines()]
                assert lines[0].startswith("s_nop 4") and lines[1].startswith("s_mov_b32 m0"), (name, lines)
                assert lines[2].startswith("s_nop 0") and lines[3].startswith("buffer_load_dwordx4"), (name, lines)
    assert n_dma > 0
