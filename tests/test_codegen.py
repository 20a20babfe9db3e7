"""Checks of the generated gfx950 code that the compiler itself cannot make.

The direct-to-LDS GEMM and row-skinny paths issue their loads as inline
assembly that sets M0 (the LDS base of a wave's 1 KB) and relies on no
compiler-generated code of those kernels keeping a value in M0; their LDS
reads are ordered after the loads by explicit waits and barriers, so every
such load must come from that assembly.  The assembly carries the one wait
state between the write of M0 and the load; the load's other hazard (five
wait states after a vector instruction writes an SGPR the load reads) is
checked here on the generated code instead of being paid with a blanket
s_nop before every load.  Compiling the sources to assembly takes a couple
of minutes on the CPU.
"""
import concurrent.futures as cf
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_19528_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


def _asm(tmp_path_factory, src):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("asm") / (src + ".s")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "--cuda-device-only", "-S",
           os.path.join(CSRC, src), "-o", str(out)]
    p = subprocess.run(cmd, capture_output=True, text=True)
    assert p.returncode == 0, p.stderr[-2000:]
    return out.read_text()


@pytest.fixture(scope="module")
def gemm_asm(tmp_path_factory):
    # the GEMM instances of both translation units (bf16 / fp32 and quantized)
    with cf.ThreadPoolExecutor(2) as ex:
        return "\n".join(ex.map(lambda src: _asm(tmp_path_factory, src), ["gemm.hip", "gemm_q.hip"]))


@pytest.fixture(scope="module")
def skinny_asm(tmp_path_factory):
    return _asm(tmp_path_factory, "skinny.hip")


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
                assert lines[0].startswith("s_mov_b32 m0") and lines[1].startswith("s_nop 0"), (name, lines)
                assert lines[2].startswith("buffer_load_dwordx4"), (name, lines)
    assert n_dma > 0


def _sgpr_hazards(asm):
    """Direct-to-LDS loads preceded, within five wait states, by a vector
    instruction that writes an SGPR of the load's resource or soffset."""
    lines = asm.splitlines()
    n, bad = 0, []
    for i, line in enumerate(lines):
        m = re.search(r"buffer_load_dwordx4\s+v\d+,\s*s\[(\d+):(\d+)\],\s*(\S+)\s+offen.*\blds\b", line)
        if not m:
            continue
        n += 1
        regs = set(range(int(m.group(1)), int(m.group(2)) + 1))
        so = m.group(3).rstrip(",")
        if re.fullmatch(r"s\d+", so):
            regs.add(int(so[1:]))
        ws, j = 0, i - 1
        while j >= 0 and ws < 5:
            t = lines[j].split(";")[0].strip()
            j -= 1
            if not t or t.startswith(".") or t.endswith(":"):
                continue
            mm = re.match(r"s_nop\s+(\d+)", t)
            if mm:
                ws += int(mm.group(1)) + 1
                continue
            d = re.match(r"v_\w+\s+(?:s\[(\d+):(\d+)\]|s(\d+)|vcc)\b", t)
            if d and (d.group(1) or d.group(3)):
                dst = {int(d.group(3))} if d.group(3) else set(range(int(d.group(1)), int(d.group(2)) + 1))
                if dst & regs:
                    bad.append((line.strip(), t))
            ws += 1
    return n, bad


def test_no_vector_written_sgpr_feeds_a_direct_to_lds_load(gemm_asm, skinny_asm):
    for asm in (gemm_asm, skinny_asm):
        n, bad = _sgpr_hazards(asm)
        assert n > 0
        assert not bad, bad[:5]


def test_hazard_scan_catches_a_planted_hazard():
    """The scan itself: a vector instruction writing the resource's SGPR right
    before the M0 write is found; three scalar instructions in between are not
    enough (five wait states)."""
    planted = "\n".join(["v_readfirstlane_b32 s9, v3", ";;#ASMSTART", "s_mov_b32 m0, s4", "s_nop 0",
                          "buffer_load_dwordx4 v1, s[8:11], s12 offen lds", ";;#ASMEND"])
    assert _sgpr_hazards(planted)[1]
    far = "\n".join(["v_readfirstlane_b32 s9, v3", "s_add_u32 s1, s1, 4", "s_add_u32 s2, s2, 4",
                      "s_add_u32 s3, s3, 4", "s_mov_b32 m0, s4", "s_nop 0",
                      "buffer_load_dwordx4 v1, s[8:11], s12 offen lds"])
    assert not _sgpr_hazards(far)[1]


def _resources(asm, name):
    tail = asm[asm.index(name + ": ;"):]
    tail = tail[tail.index(".Lfunc_end"):][:6000]
    return {k: int(re.search(r"; %s: (\d+)" % k, tail).group(1)) for k in ("ScratchSize", "NumVgprs")}


def test_gemm_kernels_make_no_calls_and_fused_backward_does_not_spill(gemm_asm):
    # A device function the compiler leaves out of line takes the kernel's
    # arguments by address, so every wave copies them to scratch memory at
    # entry.  The fused backward instances (k-major B, DMA = 2: tiles,
    # producers and side items in one kernel) must not spill at all.  (The
    # 256 x 128 row-major tiles hold 256 VGPRs per lane and spill a few
    # dwords, as measured.)
    for name, body in _kernels(gemm_asm):
        assert "s_swappc" not in body, name
        # template integers: BM BN WM WN WK BMODE BKB NBUF RD FS QB EPI DMA
        p = [int(v) for v in re.findall(r"Li(\d+)E", name)]
        assert len(p) == 13, name
        bmode, dma = p[5], p[12]
        if dma == 2 and bmode == 2:
            assert _resources(gemm_asm, name)["ScratchSize"] == 0, name
