"""GPU tests of the fused rank-r passes: producer workgroups in the GEMM
launch compute u = x A^T (forward) or du = s dy B (backward, then the dA / dB
side items) and hand them to the tiles through tagged counters in the
workspace.

The hand-over must hold when the workspace is reused by calls with other
inputs and shapes, when it starts out with arbitrary bytes, and when the same
launches are replayed from a captured graph (same tag every replay); each
result is checked against the fp64 oracle (bf16 in / fp32 accumulate,
max relative error <= 2e-2 per tensor).
"""
import sys

import pytest
import torch

from gpu_helpers import compare, oracle_lora
from workloads import lora_inputs, sample_rows

pytestmark = pytest.mark.gpu

import paper_2606_19528_amd as lm  # noqa: E402


def _announce(msg):
    print(f"[case] {msg}", file=sys.stderr, flush=True)


def _buffers(T, K, N, r):
    dev = "cuda"
    return {"y": torch.empty(T, N, dtype=torch.bfloat16, device=dev),
            "u": torch.empty(T, r, device=dev),
            "dx": torch.empty(T, K, dtype=torch.bfloat16, device=dev),
            "dA": torch.empty(r, K, device=dev), "dB": torch.empty(N, r, device=dev)}


def _step(d, o, s, ws_f, ws_b, recompute=False):
    lm.lora_linear_fwd(d["x"], d["W"], d["A"], d["B"], o["y"], o["u"], s, ws=ws_f)
    lm.lora_linear_bwd(d["x"], d["W"], d["A"], d["B"], None if recompute else o["u"], d["dy"],
                       o["dx"], o["dA"], o["dB"], s, ws=ws_b)


def _ws(T, K, N, r):
    nf = lm.lora_linear_workspace_bytes(lm.LORA_OP_FWD, T, K, N, r, lm.LORA_BF16)
    nb = lm.lora_linear_workspace_bytes(lm.LORA_OP_BWD, T, K, N, r, lm.LORA_BF16)
    n = max(nf, nb)
    return torch.empty(n, dtype=torch.uint8, device="cuda")


@pytest.mark.parametrize("shape", [(512, 1024, 1024, 16), (1000, 776, 1032, 8), (2048, 1024, 3072, 32)])
def test_reused_workspace_changing_inputs(orc, shape):
    """One workspace for every call (forward and backward share it), new inputs
    each time, and a different problem in between: every result matches the
    oracle, so no call reads rows a producer of an earlier call left behind."""
    T, K, N, r = shape
    s = 2.0
    ws = _ws(T, K, N, r)
    for it in range(4):
        _announce(f"fused reuse T={T} K={K} N={N} r={r} it={it}")
        if it == 2:
            sm = {k: v.cuda() for k, v in lora_inputs(48, 64, 128, 8, seed=90).items()}
            _step(sm, _buffers(48, 64, 128, 8), 2.0, ws, ws)
        inp = lora_inputs(T, K, N, r, seed=70 + it)
        d = {k: v.cuda() for k, v in inp.items()}
        o = _buffers(T, K, N, r)
        _step(d, o, s, ws, ws, recompute=(it == 3))
        torch.cuda.synchronize()
        rows = list(range(0, T, max(1, T // 24))) + [T - 1]
        ref = oracle_lora(orc, inp, s, rows=rows)
        compare({k: v.cpu() for k, v in o.items()}, ref, torch.bfloat16, rows=rows,
                label=f"reuse it={it}")


@pytest.mark.parametrize("fill", [0x00, 0xFF, "random"])
def test_arbitrary_workspace_contents(orc, fill):
    """The hand-over words start out as whatever the workspace holds."""
    T, K, N, r = 384, 512, 640, 16
    s = 2.0
    inp = lora_inputs(T, K, N, r, seed=81)
    d = {k: v.cuda() for k, v in inp.items()}
    ws = _ws(T, K, N, r)
    g = torch.Generator(device="cuda").manual_seed(5)
    for it in range(2):
        _announce(f"fused workspace fill={fill} it={it}")
        if fill == "random":
            ws.copy_(torch.randint(0, 256, ws.shape, dtype=torch.uint8, device="cuda", generator=g))
        else:
            ws.fill_(fill)
        o = _buffers(T, K, N, r)
        _step(d, o, s, ws, ws)
        torch.cuda.synchronize()
        ref = oracle_lora(orc, inp, s)
        compare({k: v.cpu() for k, v in o.items()}, ref, torch.bfloat16, label=f"fill={fill}")


@pytest.mark.parametrize("shape", [(256, 512, 768, 16), (1000, 1544, 1032, 12)])
def test_graph_replay(orc, shape):
    """A captured forward + backward replayed with new input values each time.
    Fused (256 x 512 -> 768): every replay carries the same tag, and each must
    still wait for its own producers (the tiles' count left by the previous
    replay keeps a stale state from passing for armed).  Unfused with the
    dA / dB items in token parts (1000 x 1544 -> 1032): the part counts the
    previous replay left must be zeroed again inside the graph."""
    T, K, N, r = shape
    s = 2.0
    rows = sample_rows(T, 64)
    d = {k: v.cuda() for k, v in lora_inputs(T, K, N, r, seed=60).items()}
    o = _buffers(T, K, N, r)
    ws_f, ws_b = _ws(T, K, N, r), _ws(T, K, N, r)
    _step(d, o, s, ws_f, ws_b)  # warm-up outside the capture
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _step(d, o, s, ws_f, ws_b)
    for it in range(4):
        _announce(f"fused graph replay it={it}")
        inp = lora_inputs(T, K, N, r, seed=61 + it)
        for k in ("x", "W", "A", "B", "dy"):
            d[k].copy_(inp[k])
        for v in o.values():
            v.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        ref = oracle_lora(orc, inp, s, rows=rows)
        compare({k: v.cpu() for k, v in o.items()}, ref, torch.bfloat16, rows=rows, label=f"replay {it}")


@pytest.mark.parametrize("shape,recompute", [((48, 2056, 1032, 8), False), ((48, 2056, 1032, 8), True),
                                             ((200, 1032, 2056, 24), False)])
def test_backward_side_items_on_producers(orc, shape, recompute):
    """Fused backward: the producers of du then run the dA / dB side items,
    here many more items than producers (3 or 13 producers, 26 items; ragged
    column blocks, rank not a multiple of 16)."""
    T, K, N, r = shape
    s = 2.0
    _announce(f"fused bwd side items T={T} K={K} N={N} r={r} recompute={recompute}")
    inp = lora_inputs(T, K, N, r, seed=95)
    d = {k: v.cuda() for k, v in inp.items()}
    ws = _ws(T, K, N, r)
    o = _buffers(T, K, N, r)
    _step(d, o, s, ws, ws, recompute=recompute)
    torch.cuda.synchronize()
    ref = oracle_lora(orc, inp, s)
    compare({k: v.cpu() for k, v in o.items()}, ref, torch.bfloat16, label="side items on producers")


def test_handover_giveup_is_reported(orc):
    """A hand-over that never completes for the tiles (the test hook makes
    their wait condition unsatisfiable) must not hang: every tile wave gives
    up after the 0.2 s budget, each kernel exits normally, and the give-ups
    are counted.  The next launches with the default settings are correct
    again and give up nowhere."""
    T, K, N, r = 384, 512, 640, 16
    p = lm.lora_linear_plan(T, K, N, r)
    assert p["fwd_fused"] and p["bwd_fused"]
    s = 2.0
    inp = lora_inputs(T, K, N, r, seed=83)
    d = {k: v.cuda() for k, v in inp.items()}
    ws = _ws(T, K, N, r)
    lm.handover_giveups(reset=True)
    try:
        lm.debug_set_handover(1)
        _announce("fused hand-over forced to give up")
        _step(d, _buffers(T, K, N, r), s, ws, ws)
        torch.cuda.synchronize()
        n = lm.handover_giveups(reset=True)
    finally:
        lm.debug_set_handover(0)
        lm.handover_giveups(reset=True)
    assert n > 0
    o = _buffers(T, K, N, r)
    _step(d, o, s, ws, ws)
    torch.cuda.synchronize()
    assert lm.handover_giveups() == 0
    ref = oracle_lora(orc, inp, s)
    compare({k: v.cpu() for k, v in o.items()}, ref, torch.bfloat16, label="after give-ups")
