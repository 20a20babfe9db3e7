"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

bf16 in / fp32 accumulate: max relative error <= 2e-2 per output tensor;
fp32 check mode: <= 1e-5.  Small shapes are compared in full; the full-size
workloads compare every element of u, dA and dB and a deterministic sample of
rows of y and dx (including the first and the last, ragged-tail, row).
"""
import os
import sys

import numpy as np
import pytest
import torch

from gpu_helpers import TOL, compare, gpu_lora, log_errors, oracle_lora, relerr
from workloads import WORKLOADS, frozen_inputs, linear_seed, lora_inputs, sample_rows

pytestmark = pytest.mark.gpu

import paper_2606_19528_amd as lm  # noqa: E402


def _announce(msg):
    print(f"[case] {msg}", file=sys.stderr, flush=True)


def _case(orc, T, K, N, r, alpha, seed=0, dtype=torch.bfloat16, rows=None, recompute=False):
    _announce(f"lora T={T} K={K} N={N} r={r} dtype={dtype} recompute={recompute}")
    s = alpha / r if r else 0.0
    inp = lora_inputs(T, K, N, r, seed=seed, dtype=dtype)
    gpu = gpu_lora(inp, s, recompute_u=recompute)
    ref = oracle_lora(orc, inp, s, rows=rows)
    return compare(gpu, ref, dtype, rows=rows, label=f"T={T} K={K} N={N} r={r}")


# --- small full-tensor cases --------------------------------------------------------
def test_single_256_full(orc):
    w = WORKLOADS["single_256"]
    lin = w.linears[0]
    _case(orc, w.tokens, lin.d_in, lin.d_out, lin.rank, lin.alpha)


@pytest.mark.parametrize("T", [1, 3, 17, 129])
@pytest.mark.parametrize("d", [8, 24, 136])
@pytest.mark.parametrize("r", [0, 1, 8, 16, 32])
def test_edge_shapes(orc, T, d, r):
    _case(orc, T, d, d + 8 * (r % 3), r, 2.0 * r if r else 0.0, seed=T * 1000 + d + r)


@pytest.mark.parametrize("shape", [(300, 520, 392, 16), (257, 392, 264, 8), (130, 1032, 136, 128),
                                   (64, 128, 2056, 5), (515, 264, 1288, 32)])
def test_multi_tile_ragged(orc, shape):
    T, K, N, r = shape
    _case(orc, T, K, N, r, 2.0 * r, seed=7)


# Shapes where the rank-r row products are split over their reduction axis
# into several partial sums (ragged last segment, up to 8 segments, odd rank,
# u rematerialised in the backward pass).
@pytest.mark.parametrize("shape,recompute,dtype", [
    ((256, 1800, 1032, 16), False, torch.bfloat16),
    ((256, 1800, 1032, 16), True, torch.bfloat16),
    ((96, 2048, 4104, 8), True, torch.bfloat16),
    ((40, 1024, 2048, 3), False, torch.bfloat16),
    ((40, 1024, 2048, 3), True, torch.bfloat16),
    ((256, 1800, 1032, 16), True, torch.float32),
])
def test_split_reduction(orc, shape, recompute, dtype):
    T, K, N, r = shape
    _case(orc, T, K, N, r, 2.0 * r, seed=41, dtype=dtype, recompute=recompute)


# Seeded random shapes over the ranges where the tile configuration, the
# fused or unfused rank-r passes, their split partial sums and the ragged
# tails change: small ones (T < 2600, d <= 3200; mostly 128 x 64 and 128 x 128
# tiles) and large ones (T >= 1024, d >= 1024; 256 x 128 to 256 x 256 tiles),
# ranks from 1 to 128.  dA and dB in full, 64 sampled rows of y and dx.
def _random_shapes(n, seed, t_range, d_range, max_macs):
    g = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        T = int(g.integers(*t_range))
        K, N = (8 * int(g.integers(d_range[0] // 8, d_range[1] // 8)) for _ in range(2))
        r = int(g.choice([1, 3, 8, 12, 16, 24, 32, 40, 64, 100, 128]))
        if T * K * N <= max_macs:
            out.append((T, K, N, r))
    return out


@pytest.mark.parametrize("shape", _random_shapes(16, 2026, (1, 2600), (8, 3200), 2.5e9) +
                         _random_shapes(10, 7, (1024, 4300), (1024, 8200), 8e10))
def test_random_shapes(orc, shape):
    T, K, N, r = shape
    _case(orc, T, K, N, r, 2.0 * r, seed=sum(shape), rows=sample_rows(T, 64))


# Long T: the rank-r row products take several 16-row tiles per workgroup, or
# whole rows, or two segments of 16-row blocks (ragged last block, rank not a
# multiple of 16, u rematerialised, reduction axes on both sides of 4096).
@pytest.mark.parametrize("shape,recompute", [((2100, 1032, 776, 24), False), ((2100, 1032, 776, 24), True),
                                             ((4100, 520, 1288, 8), True), ((2048, 3072, 1032, 32), False),
                                             ((4100, 4200, 264, 32), True), ((4100, 264, 4200, 32), False)])
def test_long_t_row_tiles(orc, shape, recompute):
    T, K, N, r = shape
    _case(orc, T, K, N, r, 2.0 * r, seed=53, recompute=recompute)


# The widest tiles (256 x 256, 32-deep stages) are picked only where they fill
# the machine in fewer waves: these shapes select them for the forward
# (d_out = 8192) and for dx (d_in = 8192), with a reduction axis that is not a
# multiple of the stage depth.  Sampled rows of y and dx; dA and dB in full.
@pytest.mark.parametrize("shape", [(4096, 264, 8192, 16), (4096, 8192, 264, 24)])
def test_wide_tiles(orc, shape):
    T, K, N, r = shape
    rows = list(range(0, T, 61)) + [T - 1]
    _case(orc, T, K, N, r, 2.0 * r, seed=59, rows=rows)


# 256 x 192 tiles fill the 256 CUs in one wave where the output is about
# 4096 x 3072: T = 4000 and d_in = d_out = 3000 select them for the forward
# (dx, which carries the dA / dB side items, runs 256 x 256 tiles; the k-major
# 256 x 192 path is covered by test_frozen_dx_one_wave_tiles), with ragged row
# and column tiles and both reduction axes not a multiple of the stage depth.
# Sampled rows of y and dx; dA and dB in full.
def test_one_wave_tiles(orc):
    T, K, N, r = 4000, 3000, 3000, 16
    p = lm.lora_linear_plan(T, K, N, r)
    assert (p["fwd_tile_m"], p["fwd_tile_n"], p["bwd_tile_m"], p["bwd_tile_n"]) == (256, 192, 256, 256)
    rows = list(range(0, T, 53)) + [T - 1]
    _case(orc, T, K, N, r, 2.0 * r, seed=61, rows=rows)


def test_split_forward_without_u_save(orc):
    # the partial sums of u stay in the workspace; y must not depend on u_save
    T, K, N, r = 256, 1800, 1032, 16
    _announce(f"fwd without u_save T={T} K={K} N={N} r={r}")
    inp = {k: v.cuda() for k, v in lora_inputs(T, K, N, r, seed=43).items()}
    y0 = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
    y1 = torch.empty_like(y0)
    u = torch.empty(T, r, dtype=torch.float32, device="cuda")
    lm.lora_linear_fwd(inp["x"], inp["W"], inp["A"], inp["B"], y0, u, 2.0)
    lm.lora_linear_fwd(inp["x"], inp["W"], inp["A"], inp["B"], y1, None, 2.0)
    torch.cuda.synchronize()
    assert torch.equal(y0, y1)
    ref = orc.u(inp["x"].cpu(), inp["A"].cpu())
    assert relerr(u.cpu().double().numpy(), ref) <= TOL[torch.bfloat16]


def test_recompute_u_matches(orc):
    T, K, N, r = 200, 264, 136, 16
    inp = lora_inputs(T, K, N, r, seed=5)
    a = gpu_lora(inp, 2.0)
    b = gpu_lora(inp, 2.0, recompute_u=True)
    for k in ("y", "dx", "dA", "dB"):
        assert torch.equal(a[k], b[k]), k


def test_deterministic(orc):
    inp = lora_inputs(333, 520, 264, 16, seed=9)
    a = gpu_lora(inp, 2.0)
    b = gpu_lora(inp, 2.0)
    for k in ("y", "dx", "u", "dA", "dB"):
        assert torch.equal(a[k], b[k]), k


# --- isolating the LoRA branch (it is only ~10% of y and dx) -----------------------
def test_zero_W_isolates_lora_branch(orc):
    T, K, N, r = 256, 384, 264, 16
    inp = lora_inputs(T, K, N, r, seed=11)
    inp["W"].zero_()
    ref = oracle_lora(orc, inp, 2.0)
    gpu = gpu_lora(inp, 2.0)
    compare(gpu, ref, torch.bfloat16, label="W=0")


def test_zero_B_gives_plain_linear(orc):
    T, K, N, r = 256, 384, 264, 16
    inp = lora_inputs(T, K, N, r, seed=12)
    inp["B"].zero_()
    gpu = gpu_lora(inp, 2.0)
    assert torch.all(gpu["dA"] == 0)
    # y must equal the rank-0 forward bitwise (the LoRA tail adds exact zeros).
    x, W = inp["x"].cuda(), inp["W"].cuda()
    y0 = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
    lm.lora_linear_fwd(x, W, None, None, y0, None, 0.0)
    torch.cuda.synchronize()
    assert torch.equal(gpu["y"], y0.cpu())
    ref = oracle_lora(orc, inp, 2.0)
    compare(gpu, ref, torch.bfloat16, label="B=0")


# --- fp32 check mode -------------------------------------------------------------
@pytest.mark.parametrize("shape", _random_shapes(8, 99, (1, 700), (8, 1100), 1e8))
def test_fp32_check_mode_random_shapes(orc, shape):
    T, K, N, r = shape
    _case(orc, T, K, N, r, 2.0 * r, seed=sum(shape), dtype=torch.float32)


@pytest.mark.parametrize("shape", [(128, 256, 256, 8), (3, 8, 24, 1), (129, 136, 144, 32),
                                   (300, 520, 392, 16), (65, 264, 128, 0)])
def test_fp32_check_mode(orc, shape):
    T, K, N, r = shape
    _case(orc, T, K, N, r, 2.0 * r if r else 0.0, seed=21, dtype=torch.float32)


# --- frozen rank-0 dx ----------------------------------------------------------------
@pytest.mark.parametrize("shape", [(1, 8, 8), (129, 136, 392), (256, 512, 1032)])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_frozen_dx_small(orc, shape, dtype):
    T, K, N = shape
    _announce(f"frozen T={T} K={K} N={N} {dtype}")
    inp = frozen_inputs(T, K, N, seed=3, dtype=dtype)
    dy, W = inp["dy"].cuda(), inp["W"].cuda()
    dx = torch.empty(T, K, dtype=dtype, device="cuda")
    lm.frozen_linear_bwd_dx(dy, W, dx)
    torch.cuda.synchronize()
    ref = orc.frozen_dx(inp["dy"], inp["W"])
    assert relerr(dx.cpu().to(torch.float64).numpy(), ref) <= TOL[dtype]


# Seeded random shapes of the frozen dx (every k-major tile shape, no side
# items): bf16 on 64 sampled rows, fp32 in full on small shapes.
@pytest.mark.parametrize("shape,dtype",
                         [(sh[:3], torch.bfloat16) for sh in _random_shapes(8, 5, (1, 4300), (8, 8200), 6e10)] +
                         [(sh[:3], torch.float32) for sh in _random_shapes(4, 6, (1, 600), (8, 1100), 1e8)])
def test_frozen_dx_random_shapes(orc, shape, dtype):
    T, K, N = shape
    _announce(f"frozen T={T} K={K} N={N} {dtype}")
    inp = frozen_inputs(T, K, N, seed=T + K + N, dtype=dtype)
    dx = torch.empty(T, K, dtype=dtype, device="cuda")
    lm.frozen_linear_bwd_dx(inp["dy"].cuda(), inp["W"].cuda(), dx)
    torch.cuda.synchronize()
    rows = sample_rows(T, 64) if dtype == torch.bfloat16 else list(range(T))
    ref = orc.frozen_dx(inp["dy"], inp["W"], rows=rows)
    assert relerr(dx.cpu().to(torch.float64).numpy()[rows], ref) <= TOL[dtype]


# 256 x 192 tiles with k-major B (frozen dx carries no side items): ragged row
# and column tiles, reduction axis not a multiple of the stage depth.
def test_frozen_dx_one_wave_tiles(orc):
    T, K, N = 4000, 3000, 1032
    _announce(f"frozen T={T} K={K} N={N}")
    inp = frozen_inputs(T, K, N, seed=5)
    dy, W = inp["dy"].cuda(), inp["W"].cuda()
    dx = torch.empty(T, K, dtype=torch.bfloat16, device="cuda")
    lm.frozen_linear_bwd_dx(dy, W, dx)
    torch.cuda.synchronize()
    rows = list(range(0, T, 37)) + [T - 1]
    ref = orc.frozen_dx(inp["dy"][rows], inp["W"])
    assert relerr(dx[rows].cpu().to(torch.float64).numpy(), ref) <= TOL[torch.bfloat16]


# --- full-size workloads (sampled rows of y and dx) --------------------------------
def _full_size(orc, key, linears=None, layer=0, fp32=False):
    w = WORKLOADS[key]
    T = w.tokens
    rows = sample_rows(T, 64)
    for idx, lin in enumerate(w.linears):
        if linears is not None and lin.name not in linears:
            continue
        dtype = torch.float32 if fp32 else torch.bfloat16
        _case(orc, T, lin.d_in, lin.d_out, lin.rank, lin.alpha, seed=linear_seed(0, layer, idx),
              dtype=dtype, rows=rows)


def test_full_llama_q_proj(orc):
    _full_size(orc, "llama_q_proj")


def test_full_llama_q_proj_fp32(orc):
    _full_size(orc, "llama_q_proj", fp32=True)


def test_full_llama_mlp(orc):
    _full_size(orc, "llama_mlp")


def test_full_qwen_layer(orc):
    _full_size(orc, "qwen_layer")


def test_full_llama_stack_layer(orc):
    # one decoder layer of the 28-layer stack (every layer has the same shapes)
    _full_size(orc, "llama_stack", layer=27)


def test_full_llama_lm_head_dx(orc):
    w = WORKLOADS["llama_stack"]
    head = w.head
    T = w.tokens
    _announce(f"lm head frozen dx T={T} K={head.d_in} N={head.d_out}")
    inp = frozen_inputs(T, head.d_in, head.d_out, seed=10_000)
    dy, W = inp["dy"].cuda(), inp["W"].cuda()
    dx = torch.empty(T, head.d_in, dtype=torch.bfloat16, device="cuda")
    lm.frozen_linear_bwd_dx(dy, W, dx)
    torch.cuda.synchronize()
    rows = sample_rows(T, 16)
    ref = orc.frozen_dx(inp["dy"][rows], inp["W"])
    err = relerr(dx.cpu()[rows].to(torch.float64).numpy(), ref)
    log_errors(f"T={T} K={head.d_in} N={head.d_out} r=0", {"dx": err})
    assert err <= TOL[torch.bfloat16]


def test_no_dw_sized_allocation():
    """The backward never allocates anything of dW's size (d_out * d_in * 2 bytes)."""
    T, K, N, r = 1024, 3072, 3072, 16
    inp = {k: v.cuda() for k, v in lora_inputs(T, K, N, r, seed=0).items()}
    ws_bytes = lm.lora_linear_workspace_bytes(lm.LORA_OP_BWD, T, K, N, r, lm.LORA_BF16)
    assert ws_bytes < N * K * 2
    u = torch.empty(T, r, device="cuda")
    y = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
    lm.lora_linear_fwd(inp["x"], inp["W"], inp["A"], inp["B"], y, u, 2.0)
    dx = torch.empty(T, K, dtype=torch.bfloat16, device="cuda")
    dA = torch.empty(r, K, device="cuda")
    dB = torch.empty(N, r, device="cuda")
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    lm.lora_linear_bwd(inp["x"], inp["W"], inp["A"], inp["B"], u, inp["dy"], dx, dA, dB, 2.0, ws=ws)
    torch.cuda.synchronize()
    assert torch.cuda.max_memory_allocated() - base == 0


def test_bwd_without_dx_matches(orc):
    """dx = NULL runs only the dA / dB reductions; they must equal the full call's."""
    T, K, N, r = 300, 264, 392, 16
    inp = {k: v.cuda() for k, v in lora_inputs(T, K, N, r, seed=31).items()}
    u = torch.empty(T, r, device="cuda")
    y = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
    lm.lora_linear_fwd(inp["x"], inp["W"], inp["A"], inp["B"], y, u, 2.0)
    outs = []
    for with_dx in (True, False):
        dx = torch.empty(T, K, dtype=torch.bfloat16, device="cuda") if with_dx else None
        dA = torch.full((r, K), float("nan"), device="cuda")
        dB = torch.full((N, r), float("nan"), device="cuda")
        lm.lora_linear_bwd(inp["x"], inp["W"], inp["A"], inp["B"], u, inp["dy"], dx, dA, dB, 2.0)
        torch.cuda.synchronize()
        outs.append((dA.cpu(), dB.cpu()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


# Where the dx tiles leave CUs idle, the dA / dB token reductions run as parts
# over consecutive token ranges and the last part of each output block adds
# the parts' tiles: two parts with a ragged second one (T = 1000: 512 + 488
# tokens), three parts (T = 1500), r = 32 (the Llama k / v case, also at full
# size in test_full_llama_stack_layer), and three parts of 1536 + 1536 + 1028
# tokens ahead of tiles that fill the CUs (T = 4100; the Llama down_proj case
# at full size in test_full_llama_stack_layer), and two rank groups (r = 40:
# 32 + 8 rank indices) in two parts.  dA and dB in full, sampled dx; then a
# second call (the counts start from zero again) and one without dx, both
# bitwise equal to the first.
@pytest.mark.parametrize("shape,parts", [((1000, 1544, 1032, 12), 2), ((1500, 1544, 2056, 12), 3),
                                         ((2000, 1544, 1032, 32), 2), ((4100, 4104, 1032, 16), 3),
                                         ((4096, 4096, 4096, 40), 2)])
def test_side_items_in_token_parts(orc, shape, parts):
    T, K, N, r = shape
    assert lm.lora_linear_plan(T, K, N, r)["bwd_side_parts"] == parts
    _case(orc, T, K, N, r, 2.0 * r, seed=61, rows=sample_rows(T, 64))
    inp = {k: v.cuda() for k, v in lora_inputs(T, K, N, r, seed=62).items()}
    u = torch.empty(T, r, device="cuda")
    y = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
    lm.lora_linear_fwd(inp["x"], inp["W"], inp["A"], inp["B"], y, u, 2.0)
    outs = []
    for with_dx in (True, True, False):
        dx = torch.empty(T, K, dtype=torch.bfloat16, device="cuda") if with_dx else None
        dA = torch.full((r, K), float("nan"), device="cuda")
        dB = torch.full((N, r), float("nan"), device="cuda")
        lm.lora_linear_bwd(inp["x"], inp["W"], inp["A"], inp["B"], u, inp["dy"], dx, dA, dB, 2.0)
        torch.cuda.synchronize()
        outs.append((dA.cpu(), dB.cpu()))
    for o in outs[1:]:
        assert torch.equal(outs[0][0], o[0]) and torch.equal(outs[0][1], o[1])


def test_repeated_calls_reuse_workspace(orc):
    """The side reductions' counters are left zeroed: back-to-back calls sharing one
    workspace (and calls with a smaller shape in between) give identical results."""
    T, K, N, r = 256, 392, 264, 32
    inp = {k: v.cuda() for k, v in lora_inputs(T, K, N, r, seed=33).items()}
    nbytes = lm.lora_linear_workspace_bytes(lm.LORA_OP_BWD, T, K, N, r, lm.LORA_BF16)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    u = torch.empty(T, r, device="cuda")
    y = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
    lm.lora_linear_fwd(inp["x"], inp["W"], inp["A"], inp["B"], y, u, 2.0)
    res = []
    for i in range(3):
        if i == 1:  # a different, smaller problem through the same workspace
            small = {k: v.cuda() for k, v in lora_inputs(40, 64, 72, 8, seed=34).items()}
            lm.lora_linear_bwd(small["x"], small["W"], small["A"], small["B"], None, small["dy"],
                               torch.empty(40, 64, dtype=torch.bfloat16, device="cuda"),
                               torch.empty(8, 64, device="cuda"), torch.empty(72, 8, device="cuda"),
                               2.0, ws=ws)
        dx = torch.empty(T, K, dtype=torch.bfloat16, device="cuda")
        dA = torch.empty(r, K, device="cuda")
        dB = torch.empty(N, r, device="cuda")
        lm.lora_linear_bwd(inp["x"], inp["W"], inp["A"], inp["B"], u, inp["dy"], dx, dA, dB, 2.0, ws=ws)
        torch.cuda.synchronize()
        res.append((dx.cpu(), dA.cpu(), dB.cpu()))
    for a, b in zip(res[0], res[2]):
        assert torch.equal(a, b)
    ref = oracle_lora(orc, {k: v.cpu() for k, v in inp.items()}, 2.0)
    compare({"dx": res[1][0], "dA": res[1][1], "dB": res[1][2]}, ref, torch.bfloat16, label="reuse")
