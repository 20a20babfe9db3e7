"""Isolation of the LoRA branch at every kernel configuration the workloads run.

The LoRA term s (x A^T) B^T is only about 7-12 % of y (and du A of dx) with
the workloads' weight scales, so a whole-tensor check of y or dx at 2e-2
would pass a LoRA branch that is off by 20 %.  Two cases isolate it:

  W = 0:  y = s u B^T and dx = du A exactly (the frozen term vanishes), so
          the LoRA-only outputs are compared with the oracle at 2e-2 of
          their own magnitude;
  B = 0:  the LoRA term adds exact zeros, so y equals the rank-0 forward
          bitwise, dA = du^T x is exactly 0 (du = s dy B = 0), and dB, u and
          dx still match the oracle.

Each shape below selects one forward and one backward configuration (GEMM
output tile, rank-r pass fused into the GEMM launch or not, one or several
partial sums of the rank-r products), asserted through lora_linear_plan; the
CPU test test_plan_coverage checks that together they cover every
configuration of every workload linear.  Sampled rows of y and dx (first
and last included), every element of u, dA and dB.
"""
import sys

import pytest
import torch

from gpu_helpers import TOL, compare, gpu_lora, oracle_lora
from workloads import lora_inputs, sample_rows

import paper_2606_19528_amd as lm  # noqa: E402

# (T, d_in, d_out, r): forward signature, backward signature, each
# (tile_m, tile_n, fused, more than one partial sum).
CASES = [
    ((128, 256, 256, 8), (128, 64, 1, 0), (128, 64, 1, 0)),
    ((1024, 3072, 3072, 16), (128, 128, 1, 0), (128, 128, 1, 0)),
    ((2048, 3072, 8192, 16), (256, 256, 0, 1), (256, 128, 1, 0)),
    ((2048, 8192, 3072, 16), (256, 128, 1, 0), (256, 256, 0, 1)),
    ((2048, 2048, 2048, 8), (128, 128, 0, 1), (128, 128, 0, 1)),
    ((2048, 2048, 11008, 8), (256, 128, 0, 1), (128, 128, 0, 1)),
    ((2048, 11008, 2048, 8), (128, 128, 0, 1), (256, 128, 0, 1)),
    ((2048, 2048, 256, 8), (128, 64, 1, 0), (128, 128, 0, 0)),
    ((4096, 3072, 3072, 32), (256, 192, 0, 0), (256, 256, 1, 0)),
    ((4096, 3072, 1024, 32), (128, 128, 0, 0), (256, 256, 0, 0)),
    ((4096, 3072, 8192, 32), (256, 256, 0, 0), (256, 256, 1, 0)),
    ((4096, 8192, 3072, 32), (256, 192, 0, 1), (256, 256, 0, 0)),
]


def signatures(T, K, N, r, dt=lm.LORA_BF16):
    p = lm.lora_linear_plan(T, K, N, r, dt)
    return ((p["fwd_tile_m"], p["fwd_tile_n"], p["fwd_fused"], int(p["fwd_u_parts"] > 1)),
            (p["bwd_tile_m"], p["bwd_tile_n"], p["bwd_fused"], int(p["bwd_du_parts"] > 1)))


def _announce(msg):
    print(f"[case] {msg}", file=sys.stderr, flush=True)


def _ids(c):
    return "x".join(str(v) for v in c[0])


@pytest.mark.gpu
@pytest.mark.parametrize("case", CASES, ids=[_ids(c) for c in CASES])
def test_zero_W_isolates_lora_branch(orc, case):
    (T, K, N, r), fwd_sig, bwd_sig = case
    assert signatures(T, K, N, r) == (fwd_sig, bwd_sig)
    _announce(f"W=0 T={T} K={K} N={N} r={r}")
    s = 2.0
    inp = lora_inputs(T, K, N, r, seed=11)
    inp["W"].zero_()
    rows = sample_rows(T, 64)
    gpu = gpu_lora(inp, s)
    ref = oracle_lora(orc, inp, s, rows=rows)
    compare(gpu, ref, torch.bfloat16, rows=rows, label=f"W=0 {T}x{K}->{N} r={r}")


@pytest.mark.gpu
@pytest.mark.parametrize("case", CASES, ids=[_ids(c) for c in CASES])
def test_zero_B_gives_plain_linear(orc, case):
    (T, K, N, r), fwd_sig, bwd_sig = case
    assert signatures(T, K, N, r) == (fwd_sig, bwd_sig)
    _announce(f"B=0 T={T} K={K} N={N} r={r}")
    s = 2.0
    inp = lora_inputs(T, K, N, r, seed=12)
    inp["B"].zero_()
    gpu = gpu_lora(inp, s)
    assert torch.all(gpu["dA"] == 0)
    x, W = inp["x"].cuda(), inp["W"].cuda()
    y0 = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
    lm.lora_linear_fwd(x, W, None, None, y0, None, 0.0)
    torch.cuda.synchronize()
    assert torch.equal(gpu["y"], y0.cpu())
    rows = sample_rows(T, 64)
    ref = oracle_lora(orc, inp, s, rows=rows)
    compare(gpu, ref, torch.bfloat16, rows=rows, label=f"B=0 {T}x{K}->{N} r={r}")


@pytest.mark.gpu
@pytest.mark.parametrize("shape", [(300, 520, 392, 16), (129, 136, 144, 32)])
def test_zero_W_fp32_check_mode(orc, shape):
    T, K, N, r = shape
    _announce(f"W=0 fp32 T={T} K={K} N={N} r={r}")
    inp = lora_inputs(T, K, N, r, seed=13, dtype=torch.float32)
    inp["W"].zero_()
    gpu = gpu_lora(inp, 2.0)
    ref = oracle_lora(orc, inp, 2.0)
    errs = compare(gpu, ref, torch.float32, label=f"W=0 fp32 {shape}")
    assert max(errs.values()) <= TOL[torch.float32]
