"""GPU checks of the checkpointed step over a chain of LoRA linears: its
outputs and gradients are bitwise those of the plain chain of lora_linear_fwd
/ lora_linear_bwd calls (same kernels, u saved instead of recomputed) and
within the bf16 tolerance of the fp64 oracle's chain; with separate compute
and copy streams and with one stream for both."""
import sys

import pytest
import torch

from gpu_helpers import TOL, relerr
from workloads import lora_inputs

pytestmark = pytest.mark.gpu

import paper_2606_19528_amd as lm  # noqa: E402


def _announce(msg):
    print(f"[case] {msg}", file=sys.stderr, flush=True)


def _chain_inputs(T, dims, ranks, seed):
    nodes = []
    for i in range(len(dims) - 1):
        inp = lora_inputs(T, dims[i], dims[i + 1], ranks[i], seed=seed + i)
        nodes.append({"W": inp["W"].cuda(), "A": inp["A"].cuda(), "B": inp["B"].cuda(),
                      "scale": 2.0 if ranks[i] else 0.0,
                      "dA": torch.empty(ranks[i], dims[i], device="cuda"),
                      "dB": torch.empty(dims[i + 1], ranks[i], device="cuda")})
    first = lora_inputs(T, dims[0], dims[-1], 1, seed=seed + 100)
    return nodes, first["x"].cuda(), first["dy"].cuda()


def _plain(nodes, x0, g):
    xs = [x0]
    us = []
    for nd in nodes:
        y = torch.empty(x0.shape[0], nd["W"].shape[0], dtype=torch.bfloat16, device="cuda")
        u = torch.empty(x0.shape[0], nd["A"].shape[0], dtype=torch.float32, device="cuda")
        lm.lora_linear_fwd(xs[-1], nd["W"], nd["A"], nd["B"], y, u, nd["scale"])
        xs.append(y)
        us.append(u)
    grads = []
    for i in range(len(nodes) - 1, -1, -1):
        nd = nodes[i]
        dx = torch.empty_like(xs[i])
        dA, dB = torch.empty_like(nd["dA"]), torch.empty_like(nd["dB"])
        lm.lora_linear_bwd(xs[i], nd["W"], nd["A"], nd["B"], us[i], g, dx, dA, dB, nd["scale"])
        grads.insert(0, (dA, dB))
        g = dx
    torch.cuda.synchronize()
    return xs[-1], grads, g


@pytest.mark.parametrize("streams", ["two", "one"])
@pytest.mark.parametrize("case", [
    (129, [256, 512, 256, 392], [8, 16, 5]),
    (300, [1024, 3072, 1024, 3072, 1024], [16, 16, 16, 16]),
])
def test_ckpt_chain(orc, case, streams):
    T, dims, ranks = case
    _announce(f"ckpt T={T} dims={dims} ranks={ranks} streams={streams}")
    nodes, x0, g = _chain_inputs(T, dims, ranks, seed=T)
    ws_b, host_b = lm.lora_ckpt_sizes(nodes, T)
    ws = torch.empty(ws_b, dtype=torch.uint8, device="cuda")
    stash = torch.empty(host_b, dtype=torch.uint8, pin_memory=True)
    cs = torch.cuda.Stream()
    xs_ = torch.cuda.Stream() if streams == "two" else cs
    out = torch.empty(T, dims[-1], dtype=torch.bfloat16, device="cuda")
    dx0 = torch.empty(T, dims[0], dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    lm.lora_ckpt_forward(nodes, x0, out, stash, ws, cs, xs_)
    lm.lora_ckpt_backward(nodes, g, dx0, stash, ws, cs, xs_)
    torch.cuda.synchronize()
    ref_out, ref_grads, ref_dx0 = _plain(nodes, x0, g)
    assert torch.equal(out, ref_out)
    assert torch.equal(dx0, ref_dx0)
    for nd, (dA, dB) in zip(nodes, ref_grads):
        assert torch.equal(nd["dA"], dA) and torch.equal(nd["dB"], dB)
    # against the fp64 oracle's chain
    on = [{"W": nd["W"].cpu(), "A": nd["A"].cpu(), "B": nd["B"].cpu(), "s": nd["scale"]} for nd in nodes]
    oxs, ograds, odx0 = orc.chain(x0.cpu(), on, g.cpu())
    tol = TOL[torch.bfloat16]
    errs = [relerr(out.cpu().double().numpy(), oxs[-1]), relerr(dx0.cpu().double().numpy(), odx0)]
    for nd, og in zip(nodes, ograds):
        errs += [relerr(nd["dA"].cpu().double().numpy(), og["dA"]),
                 relerr(nd["dB"].cpu().double().numpy(), og["dB"])]
    _announce(f"  max rel err {max(errs):.2e}")
    assert max(errs) <= tol, errs


def test_ckpt_stash_holds_the_inputs(orc):
    # the host stash holds every node's input, in order, after the forward
    T, dims, ranks = 64, [256, 384, 256], [8, 8]
    nodes, x0, g = _chain_inputs(T, dims, ranks, seed=7)
    ws_b, host_b = lm.lora_ckpt_sizes(nodes, T)
    ws = torch.empty(ws_b, dtype=torch.uint8, device="cuda")
    stash = torch.empty(host_b, dtype=torch.uint8, pin_memory=True)
    out = torch.empty(T, dims[-1], dtype=torch.bfloat16, device="cuda")
    lm.lora_ckpt_forward(nodes, x0, out, stash, ws, torch.cuda.current_stream(), torch.cuda.Stream())
    torch.cuda.synchronize()
    x1 = torch.empty(T, dims[1], dtype=torch.bfloat16, device="cuda")
    lm.lora_linear_fwd(x0, nodes[0]["W"], nodes[0]["A"], nodes[0]["B"], x1, None, nodes[0]["scale"])
    torch.cuda.synchronize()
    n0 = T * dims[0] * 2
    assert torch.equal(stash[:n0].view(torch.bfloat16).view(T, dims[0]), x0.cpu())
    assert torch.equal(stash[n0:n0 + T * dims[1] * 2].view(torch.bfloat16).view(T, dims[1]), x1.cpu())
