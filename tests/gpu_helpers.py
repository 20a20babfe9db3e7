"""Shared helpers for the GPU parity tests: run the HIP path through the C ABI
and compare with the fp64 oracle.

Error metric (per tensor): max_i |gpu_i - ref_i| / max_i |ref_i|, the
definition of "max relative error" used throughout the tests; an elementwise
ratio would blow up where the reference is near zero.
"""
from __future__ import annotations

import json
import os

import numpy as np
import torch

import paper_2606_19528_amd as lm

TOL = {torch.bfloat16: 2e-2, torch.float32: 1e-5}


def relerr(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    den = float(np.max(np.abs(ref)))
    num = float(np.max(np.abs(got - ref)))
    return num / den if den > 0 else num


def to_dev(inp: dict) -> dict:
    return {k: v.to("cuda") for k, v in inp.items()}


def gpu_lora(inp: dict, s: float, recompute_u: bool = False, want_dx: bool = True) -> dict:
    """Forward then backward of one LoRA linear on cuda:0 through the C ABI.
    `inp` holds CPU or GPU tensors x, W, A, B, dy; returns CPU tensors."""
    d = {k: v.to("cuda") for k, v in inp.items()}
    x, W, A, B, dy = d["x"], d["W"], d["A"], d["B"], d["dy"]
    T, K = x.shape
    N = W.shape[0]
    r = A.shape[0]
    dt = x.dtype
    y = torch.empty(T, N, dtype=dt, device="cuda")
    u = torch.empty(T, r, dtype=torch.float32, device="cuda") if r else None
    lm.lora_linear_fwd(x, W, A if r else None, B if r else None, y, u, s)
    dx = torch.empty(T, K, dtype=dt, device="cuda") if want_dx else None
    dA = torch.empty(r, K, dtype=torch.float32, device="cuda") if r else None
    dB = torch.empty(N, r, dtype=torch.float32, device="cuda") if r else None
    lm.lora_linear_bwd(x, W, A if r else None, B if r else None, None if recompute_u else u, dy,
                       dx, dA, dB, s)
    torch.cuda.synchronize()
    out = {"y": y.cpu(), "dx": dx.cpu() if want_dx else None}
    if r:
        out.update(u=u.cpu(), dA=dA.cpu(), dB=dB.cpu())
    return out


def gpu_lora_q(inp: dict, Wq: dict, s: float, recompute_u: bool = False) -> dict:
    """gpu_lora with the frozen W given quantized (workloads.quant_weight);
    inp["W"] is ignored."""
    d = {k: v.to("cuda") for k, v in inp.items() if k != "W"}
    q = {k: (v.to("cuda") if hasattr(v, "to") else v) for k, v in Wq.items()}
    x, A, B, dy = d["x"], d["A"], d["B"], d["dy"]
    T, K = x.shape
    N = dy.shape[1]
    r = A.shape[0]
    y = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
    u = torch.empty(T, r, dtype=torch.float32, device="cuda") if r else None
    lm.lora_linear_fwd_q(x, q, A if r else None, B if r else None, y, u, s)
    dx = torch.empty(T, K, dtype=torch.bfloat16, device="cuda")
    dA = torch.empty(r, K, dtype=torch.float32, device="cuda") if r else None
    dB = torch.empty(N, r, dtype=torch.float32, device="cuda") if r else None
    lm.lora_linear_bwd_q(x, q, A if r else None, B if r else None, None if recompute_u else u, dy,
                         dx, dA, dB, s)
    torch.cuda.synchronize()
    out = {"y": y.cpu(), "dx": dx.cpu()}
    if r:
        out.update(u=u.cpu(), dA=dA.cpu(), dB=dB.cpu())
    return out


def oracle_lora(orc, inp: dict, s: float, rows=None) -> dict:
    """Oracle results; y and dx restricted to `rows` (all rows if None)."""
    x, W, A, B, dy = (inp[k] for k in ("x", "W", "A", "B", "dy"))
    U = orc.u(x, A)
    G, dU = orc.grad_u(dy, B, s)
    return {"u": U, "y": orc.y(x, W, U, B, s, rows=rows), "dx": orc.dx(dy, W, dU, A, rows=rows),
            "dA": orc.da(dU, x), "dB": orc.db(dy, U, s)}


def log_errors(label: str, errs: dict) -> None:
    """Append the errors of one case to the JSON-lines file named by
    LORA_PARITY_LOG, if set (a record of the achieved errors per test)."""
    path = os.environ.get("LORA_PARITY_LOG")
    if not path:
        return
    test = os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]
    with open(path, "a") as f:
        f.write(json.dumps({"test": test, "case": label, "errors": errs}) + "\n")


def compare(gpu: dict, ref: dict, dtype, rows=None, label: str = "") -> dict:
    """Per-tensor errors; asserts each is within the dtype's tolerance."""
    tol = TOL[dtype]
    errs = {}
    for k in ("y", "dx", "u", "dA", "dB"):
        if k not in ref or gpu.get(k) is None:
            continue
        g = gpu[k].to(torch.float64).numpy()
        if rows is not None and k in ("y", "dx"):
            g = g[rows]
        errs[k] = relerr(g, ref[k])
    log_errors(label, errs)
    bad = {k: e for k, e in errs.items() if not e <= tol}
    assert not bad, f"{label} errors above {tol}: {bad} (all: {errs})"
    return errs
