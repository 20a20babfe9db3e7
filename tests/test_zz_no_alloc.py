"""lora_linear_bwd_noalloc: the backward with the library's static device
scratch as workspace, for callers that cannot allocate.  Checked against
lora_linear_bwd (the same kernels with a caller workspace) through the C ABI:
every output bitwise equal and within the fp64 oracle's tolerance, on calls
in a row whose later ones use smaller inputs (the scratch keeps the
previous call's contents), with no device allocation during the calls; and,
on the CPU, the rejection of sizes beyond the scratch.
"""
import ctypes
import sys

import pytest
import torch

from gpu_helpers import compare, oracle_lora
from workloads import lora_inputs, sample_rows

import paper_2606_19528_amd as lm
from paper_2606_19528_amd import lora as L


def P(i):
    return ctypes.c_void_p(0x7F0000000000 + i * 0x100000000)


def test_noalloc_rejects_sizes_beyond_the_scratch():
    """Sizes whose workspace exceeds the static scratch: LORA_EWORKSPACE before
    any device work (fake, never-dereferenced pointers)."""
    T, K, N, r = 65536, 8192, 8192, 128
    assert lm.lora_linear_workspace_bytes(L.LORA_OP_BWD, T, K, N, r, L.LORA_BF16) > 16 << 20
    lib = lm.lib()
    st = lib.lora_linear_bwd_noalloc(P(1), P(2), P(3), P(4), P(6), P(8), P(9), P(10), P(11), T, K, N, r,
                                     2.0, L.LORA_BF16, None)
    assert st == L.LORA_EWORKSPACE
    assert b"static scratch" in lib.lora_last_error()
    # sizes the entry point rejects anyway report the usual code
    st = lib.lora_linear_bwd_noalloc(P(1), P(2), P(3), P(4), P(6), P(8), P(9), P(10), P(11), 64, 250, 256,
                                     8, 2.0, L.LORA_BF16, None)
    assert st == L.LORA_EUNSUPPORTED


def _bufs(T, K, N, r, dev="cuda"):
    return (torch.empty(T, K, dtype=torch.bfloat16, device=dev), torch.empty(r, K, device=dev),
            torch.empty(N, r, device=dev))


@pytest.mark.gpu
def test_noalloc_matches_workspace_entry_point(orc):
    # fused backward (q_proj), an unfused one with split partial sums, one
    # whose dA / dB items run as token parts (their counts must start from
    # zero in a scratch that holds the previous call's), then a smaller fused
    # one: each after the previous left its state in the scratch
    shapes = [(1024, 3072, 3072, 16), (2048, 2048, 2048, 8), (1000, 1544, 1032, 12), (300, 520, 392, 16)]
    assert lm.lora_linear_plan(1000, 1544, 1032, 12)["bwd_side_parts"] == 2
    for i, (T, K, N, r) in enumerate(shapes):
        print(f"[case] noalloc bwd T={T} K={K} N={N} r={r}", file=sys.stderr, flush=True)
        s = 2.0
        inp = lora_inputs(T, K, N, r, seed=200 + i)
        d = {k: v.cuda() for k, v in inp.items()}
        u = torch.empty(T, r, device="cuda")
        y = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
        lm.lora_linear_fwd(d["x"], d["W"], d["A"], d["B"], y, u, s)
        ref_out = _bufs(T, K, N, r)
        lm.lora_linear_bwd(d["x"], d["W"], d["A"], d["B"], u, d["dy"], *ref_out, s)
        got = _bufs(T, K, N, r)
        for t in got:
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        st = lm.lib().lora_linear_bwd_noalloc(
            L._ptr(d["x"]), L._ptr(d["W"]), L._ptr(d["A"]), L._ptr(d["B"]), L._ptr(u), L._ptr(d["dy"]),
            L._ptr(got[0]), L._ptr(got[1]), L._ptr(got[2]), T, K, N, r, s, L.LORA_BF16,
            L._stream(None))
        assert st == L.LORA_OK, lm.lib().lora_last_error()
        torch.cuda.synchronize()
        assert torch.cuda.max_memory_allocated() == base
        for a, b in zip(ref_out, got):
            assert torch.equal(a, b)
        rows = sample_rows(T, 64)
        ref = oracle_lora(orc, inp, s, rows=rows)
        compare({"dx": got[0].cpu(), "dA": got[1].cpu(), "dB": got[2].cpu()}, ref, torch.bfloat16,
                rows=rows, label=f"noalloc {T}x{K}->{N}")
