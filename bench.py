"""Benchmark of the LoRA-linear hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step = the forward of every LoRA linear of the workload, then the
backward of each in reverse order (u saved by the forward is reused), plus the
frozen LM head's dx when the workload has one.  Inputs are synthetic (seeded
Gaussian, bf16) and resident in HBM before timing starts.  Prints one JSON
line: throughput in TFLOP/s of algorithmic work (4TKN + 6Tr(K+N) per LoRA
linear, 2TKN per frozen dx), the dominant kernel's roofline position measured
with HIP events around its launches, peak workspace bytes, and the fp64 CPU
oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2606_19528_amd as lm  # noqa: E402
from workloads import (ORDER, WORKLOADS, frozen_inputs, head_inputs, linear_seed,  # noqa: E402
                       lora_inputs, quant_weight)

METRIC = "LoRA linear fwd+bwd TFLOP/s (% bf16 MFMA peak) + peak device workspace bytes"
PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 4096 dense bf16 flop/clk x 2.4 GHz
PEAK_HBM_GBS = 8000.0


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_sha():
    """Hash of the kernel sources: a stored counter measurement is only used
    while the code it was taken on is unchanged."""
    import hashlib

    d = os.path.join(ROOT, "paper_2606_19528_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(os.listdir(d)):
        if name.endswith((".hip", ".hpp", ".cpp", ".h")):
            h.update(name.encode())
            with open(os.path.join(d, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()[:16]


def stored_traffic(workload_key):
    """HBM-side bytes per launch of each library kernel from the committed
    counter summary (FETCH_SIZE + WRITE_SIZE, calibrated against a copy of
    known size), or {} when it was taken on other code or another workload."""
    path = os.path.join(ROOT, "profiles", f"lora_linear_{workload_key}_traffic.md")
    if not os.path.exists(path):
        return {}
    meta = {}
    with open(path) as f:
        for line in f:
            if line.startswith("<!-- ") and ":" in line:
                k, v = line[5:].rstrip().rstrip(">").rstrip("-").strip().split(":", 1)
                meta[k.strip()] = v.strip()
    if meta.get("source_sha") != kernel_source_sha() or meta.get("workload") != workload_key:
        return {}
    try:
        return {k: int(v) for k, v in json.loads(meta.get("traffic_bytes_per_launch", "{}")).items()}
    except ValueError:
        return {}


class Layer:
    """Device buffers of one LoRA linear (inputs, outputs, workspace)."""

    def __init__(self, lin, T, seed, dev):
        self.lin = lin
        K, N, r = lin.d_in, lin.d_out, lin.rank
        inp = lora_inputs(T, K, N, r, seed=seed, device=dev)
        self.x, self.W, self.A, self.B, self.dy = (inp[k] for k in ("x", "W", "A", "B", "dy"))
        self.y = torch.empty(T, N, dtype=torch.bfloat16, device=dev)
        self.u = torch.empty(T, r, dtype=torch.float32, device=dev)
        self.dx = torch.empty(T, K, dtype=torch.bfloat16, device=dev)
        self.dA = torch.empty(r, K, dtype=torch.float32, device=dev)
        self.dB = torch.empty(N, r, dtype=torch.float32, device=dev)
        self.T = T


def build(workload, dev):
    T = workload.tokens
    layers = []
    for layer in range(workload.layers):
        for idx, lin in enumerate(workload.linears):
            layers.append(Layer(lin, T, linear_seed(0, layer, idx), dev))
    head = None
    if workload.head is not None:
        h = workload.head
        hi = frozen_inputs(T, h.d_in, h.d_out, seed=10_000, device=dev)
        head = (hi["dy"], hi["W"], torch.empty(T, h.d_in, dtype=torch.bfloat16, device=dev))
    ws_bytes = 0
    for L in layers:
        K, N, r = L.lin.d_in, L.lin.d_out, L.lin.rank
        ws_bytes = max(ws_bytes,
                       lm.lora_linear_workspace_bytes(lm.LORA_OP_FWD, T, K, N, r, lm.LORA_BF16),
                       lm.lora_linear_workspace_bytes(lm.LORA_OP_BWD, T, K, N, r, lm.LORA_BF16))
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    return layers, head, ws, ws_bytes


def step(layers, head, ws):
    for L in layers:
        lm.lora_linear_fwd(L.x, L.W, L.A, L.B, L.y, L.u, L.lin.scale, ws=ws)
    if head is not None:
        lm.frozen_linear_bwd_dx(head[0], head[1], head[2])
    for L in reversed(layers):
        lm.lora_linear_bwd(L.x, L.W, L.A, L.B, L.u, L.dy, L.dx, L.dA, L.dB, L.lin.scale, ws=ws)


def build_quant(layers, head, workload, dev):
    """INT4 codes (groups of 128 inputs) for every LoRA linear's frozen W and
    INT8 codes for the frozen head, the paper's mixed-precision setting."""
    qs = [quant_weight(L.lin.d_out, L.lin.d_in, 4, 128, seed=1000 + i, device=dev)
          for i, L in enumerate(layers)]
    qh = None
    if head is not None:
        h = workload.head
        qh = quant_weight(h.d_out, h.d_in, 8, 128, seed=20_000, device=dev)
    return qs, qh


def step_quant(layers, head, ws, qs, qh):
    for L, q in zip(layers, qs):
        lm.lora_linear_fwd_q(L.x, q, L.A, L.B, L.y, L.u, L.lin.scale, ws=ws)
    if head is not None:
        lm.frozen_linear_bwd_dx_q(head[0], qh, head[2])
    for L, q in zip(reversed(layers), reversed(qs)):
        lm.lora_linear_bwd_q(L.x, q, L.A, L.B, L.u, L.dy, L.dx, L.dA, L.dB, L.lin.scale, ws=ws)


def time_steps(fn, steps, warmup):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def percentiles(v):
    """median, p10, p90 of a list of step times (ms)."""
    t = torch.tensor(sorted(v), dtype=torch.float64)
    q = torch.quantile(t, torch.tensor([0.5, 0.1, 0.9], dtype=torch.float64))
    return {"median_ms": round(float(q[0]), 5), "p10_ms": round(float(q[1]), 5),
            "p90_ms": round(float(q[2]), 5)}


def event_steps(fn, steps, flush=None):
    """Run `steps` steps with an event between consecutive steps; with `flush`
    (a device buffer) every step is preceded, outside its own event pair, by a
    write of the whole buffer, which evicts the 256 MB last-level cache (the
    cold-cache protocol).  Returns (total ms from first to last event, list of
    per-step ms)."""
    n = steps + 1 if flush is None else 2 * steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
    torch.cuda.synchronize()
    if flush is None:
        ev[0].record()
        for i in range(steps):
            fn()
            ev[i + 1].record()
    else:
        for i in range(steps):
            flush.fill_(i & 0xFF)
            ev[2 * i].record()
            fn()
            ev[2 * i + 1].record()
    torch.cuda.synchronize()
    if flush is None:
        per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
        return ev[0].elapsed_time(ev[steps]), per
    per = [ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(steps)]
    return sum(per), per


def per_kernel_ms(fn, steps):
    lm.profiler_reset()
    lm.profiler_enable(True)
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    lm.profiler_enable(False)
    out = {}
    for name in lm.kernel_names():
        tot, n = lm.profiler_read(name)
        if n:
            out[name] = (tot, n)
    lm.profiler_reset()
    return out


def algorithmic(workload):
    """Algorithmic work of one step per library kernel, from the plan of each
    linear (which GEMM launches carry the rank-r producers, which products run
    as separate row-skinny launches).  GEMM launches: flops (the dx launch also
    does the dA / dB token reductions, 2Tr(K+N)).  Row-skinny launches: the
    bytes they must move (inputs once, fp32 outputs once) and their flops.
      forward   gemm_fwd     2TN(K+r) (+ 2TKr when u = x A^T runs inside it)
                lora_down    2TK + 2rK + 4Tr bytes, 2TKr flops (otherwise)
      backward  gemm_bwd_dx  2TK(N+r) + 2Tr(K+N) (+ 2TNr when du = s dy B runs inside it)
                lora_dy_b    2TN + 2Nr + 4Tr bytes, 2TNr flops (otherwise)
      head      gemm_frozen_dx  2TKN"""
    T = workload.tokens
    flops, nbytes = {}, {}

    def add(d, k, v):
        d[k] = d.get(k, 0.0) + v

    for lin in workload.linears:
        K, N, r = lin.d_in, lin.d_out, lin.rank
        p = lm.lora_linear_plan(T, K, N, r)
        L = workload.layers
        add(flops, "gemm_fwd", L * (2.0 * T * N * (K + r) + (2.0 * T * K * r if p["fwd_fused"] else 0.0)))
        if not p["fwd_fused"]:
            add(flops, "lora_down", L * 2.0 * T * K * r)
            add(nbytes, "lora_down", L * (2.0 * T * K + 2.0 * r * K + 4.0 * T * r))
        add(flops, "gemm_bwd_dx", L * (2.0 * T * K * (N + r) + 2.0 * T * r * (K + N)
                                       + (2.0 * T * N * r if p["bwd_fused"] else 0.0)))
        if not p["bwd_fused"]:
            add(flops, "lora_dy_b", L * 2.0 * T * N * r)
            add(nbytes, "lora_dy_b", L * (2.0 * T * N + 2.0 * N * r + 4.0 * T * r))
    if workload.head is not None:
        add(flops, "gemm_frozen_dx", 2.0 * T * workload.head.d_in * workload.head.d_out)
    return flops, nbytes


def kernel_table(workload, per_kernel, steps):
    """Per library kernel: time per step, launches, average launch, and the
    roofline position (TFLOP/s against the dense bf16 peak for the GEMMs, GB/s
    of algorithmic bytes against HBM for the row-skinny kernels)."""
    flops, nbytes = algorithmic(workload)
    out = {}
    for name, (tot, n) in per_kernel.items():
        ms = tot / steps
        e = {"ms_per_step": round(ms, 5), "launches_per_step": round(n / steps, 3),
             "avg_launch_us": round(tot / n * 1e3, 3)}
        if name in nbytes:
            gbs = nbytes[name] / (ms * 1e-3) / 1e9
            e.update({"bound": "hbm", "achieved": round(gbs, 1), "unit": "GB/s",
                      "frac": round(gbs / PEAK_HBM_GBS, 4),
                      "bytes_per_launch": round(nbytes[name] / (n / steps))})
        elif name in flops:
            tf = flops[name] / (ms * 1e-3) / 1e12
            e.update({"bound": "mfma", "achieved": round(tf, 2), "unit": "TFLOP/s",
                      "frac": round(tf / PEAK_BF16_TFLOPS, 4),
                      "flops_per_launch": round(flops[name] / (n / steps))})
        out[name] = e
    return out


def bench_lm_head(dev, steps=5, warmup=2, T=4096, V=128256, D=3072, k=1000, trainable=0.3):
    """The frozen LM head of the 3B model at the paper's top-1000 / 30 %
    trainable setting: reduced vocabulary J, then loss and dh over the
    trainable positions only; beside it the full-vocabulary head over every
    position (the same kernels with J = [0, V) and all rows), which is what
    the reduction avoids."""
    d = {k_: v.to(dev) for k_, v in head_inputs(T, V, D, k, trainable, seed=3).items()}
    nrows = d["rows"].numel()
    J, tpos = lm.lm_head_build_vocab(d["table"], k, d["targets"], d["rows"])
    nJ = J.numel()
    loss = torch.empty(T, dtype=torch.float32, device=dev)
    total = torch.empty(1, dtype=torch.float32, device=dev)
    dh = torch.empty(T, D, dtype=torch.bfloat16, device=dev)
    ws = torch.empty(lm.lm_head_workspace_bytes(2, T, V, D, T, V), dtype=torch.uint8, device=dev)
    wsv = torch.empty(lm.lm_head_workspace_bytes(0, T, V, D, nrows), dtype=torch.uint8, device=dev)
    t0 = time.perf_counter()
    for _ in range(steps):
        lm.lm_head_build_vocab(d["table"], k, d["targets"], d["rows"], ws=wsv)
    ms_vocab = (time.perf_counter() - t0) / steps * 1e3   # includes the wait for |J|
    red = lambda: lm.lm_head_reduced_ce(d["h"], d["W"], d["rows"], J, tpos, loss[:nrows],  # noqa: E731
                                        total, dh, 1.0, ws=ws)
    ms_red = time_steps(red, steps, warmup)
    allrows = torch.arange(T, dtype=torch.int32, device=dev)
    Jall = torch.arange(V, dtype=torch.int32, device=dev)
    tall = d["targets"]
    full = lambda: lm.lm_head_reduced_ce(d["h"], d["W"], allrows, Jall, tall, loss, total, dh,  # noqa: E731
                                         1.0, ws=ws)
    ms_full = time_steps(full, 2, 1)
    fl_red = 6.0 * nrows * nJ * D
    return {"T": T, "V": V, "D": D, "k": k, "trainable_positions": nrows, "reduced_vocab": nJ,
            "ms_build_vocab": round(ms_vocab, 4), "ms_loss_and_dh": round(ms_red, 4),
            "tflops_loss_and_dh": round(fl_red / (ms_red * 1e-3) / 1e12, 2),
            "ms_full_vocab_all_positions": round(ms_full, 4),
            "tflops_full": round(6.0 * T * V * D / (ms_full * 1e-3) / 1e12, 2)}


def bench_ckpt(dev, T=2048, pairs=4, d=3072, h=8192, r=16, steps=5, warmup=2):
    """A chain of 2*pairs LoRA linears d -> h -> d -> ... (the MLP shapes of the
    3B model) run plainly (every node's input and u kept on the device) and
    checkpointed (inputs offloaded to pinned host memory over PCIe, u
    recomputed): time per fwd+bwd and the device bytes each keeps."""
    dims = [d, h] * pairs + [d]
    nodes = []
    for i in range(len(dims) - 1):
        inp = lora_inputs(T, dims[i], dims[i + 1], r, seed=500 + i, device=dev)
        nodes.append({"W": inp["W"], "A": inp["A"], "B": inp["B"], "scale": 2.0,
                      "dA": torch.empty(r, dims[i], device=dev),
                      "dB": torch.empty(dims[i + 1], r, device=dev)})
    x0 = torch.randn(T, d, device=dev).to(torch.bfloat16)
    g = torch.randn(T, d, device=dev).to(torch.bfloat16)
    # plain: all activations and u resident
    xs = [x0] + [torch.empty(T, dims[i + 1], dtype=torch.bfloat16, device=dev) for i in range(len(nodes))]
    us = [torch.empty(T, r, device=dev) for _ in nodes]
    gbuf = [torch.empty(T * max(dims), dtype=torch.bfloat16, device=dev) for _ in range(2)]
    wsz = max(max(lm.lora_linear_workspace_bytes(o, T, dims[i], dims[i + 1], r, lm.LORA_BF16)
                  for o in (0, 1)) for i in range(len(nodes)))
    ws = torch.empty(wsz, dtype=torch.uint8, device=dev)

    def plain():
        for i, nd in enumerate(nodes):
            lm.lora_linear_fwd(xs[i], nd["W"], nd["A"], nd["B"], xs[i + 1], us[i], 2.0, ws=ws)
        gi = g
        for i in range(len(nodes) - 1, -1, -1):
            nd = nodes[i]
            dx = gbuf[i % 2][: T * dims[i]].view(T, dims[i])
            lm.lora_linear_bwd(xs[i], nd["W"], nd["A"], nd["B"], us[i], gi, dx, nd["dA"], nd["dB"],
                               2.0, ws=ws)
            gi = dx

    ms_plain = time_steps(plain, steps, warmup)
    plain_bytes = sum(x.numel() * 2 for x in xs[1:]) + sum(u.numel() * 4 for u in us) + \
        sum(b.numel() * 2 for b in gbuf) + wsz
    cw, ch = lm.lora_ckpt_sizes(nodes, T)
    cws = torch.empty(cw, dtype=torch.uint8, device=dev)
    stash = torch.empty(ch, dtype=torch.uint8, pin_memory=True)
    out = torch.empty(T, d, dtype=torch.bfloat16, device=dev)
    dx0 = torch.empty(T, d, dtype=torch.bfloat16, device=dev)
    cs, cp = torch.cuda.current_stream(), torch.cuda.Stream()

    def ckpt():
        lm.lora_ckpt_forward(nodes, x0, out, stash, cws, cs, cp)
        lm.lora_ckpt_backward(nodes, g, dx0, stash, cws, cs, cp)

    ms_ckpt = time_steps(ckpt, steps, warmup)
    torch.cuda.synchronize()
    flops = sum(4.0 * T * dims[i] * dims[i + 1] + 6.0 * T * r * (dims[i] + dims[i + 1])
                for i in range(len(nodes)))
    return {"T": T, "nodes": len(nodes), "dims": dims, "rank": r,
            "ms_plain": round(ms_plain, 4), "ms_checkpointed": round(ms_ckpt, 4),
            "tflops_plain": round(flops / (ms_plain * 1e-3) / 1e12, 2),
            "tflops_checkpointed": round(flops / (ms_ckpt * 1e-3) / 1e12, 2),
            "device_bytes_plain": int(plain_bytes), "device_bytes_checkpointed": int(cw + 2 * out.numel() * 2),
            "host_stash_bytes": int(ch)}


def bench_topk(dev, V=128256, D=3072, k=1000):
    """The similarity table of the 3B model's output embedding (k = 1000):
    one build, after one warm-up build; the work is the V x V x D similarity
    GEMM (the selection streams behind it)."""
    W = (torch.randn(V, D, device=dev) * 0.02).to(torch.bfloat16)
    table = torch.empty(V, k, dtype=torch.int32, device=dev)
    ws = torch.empty(lm.lora.lib().topk_table_workspace_bytes(V, D, k), dtype=torch.uint8, device=dev)
    ms = time_steps(lambda: lm.topk_table_build(W, k, table, ws=ws), 1, 1)
    pk = per_kernel_ms(lambda: lm.topk_table_build(W, k, table, ws=ws), 1)
    return {"V": V, "D": D, "k": k, "ms": round(ms, 2),
            "tflops_similarity": round(2.0 * V * V * D / (ms * 1e-3) / 1e12, 2),
            "kernels_ms": {n: round(v[0], 2) for n, v in pk.items()},
            "table_bytes": V * k * 4}


def cpu_info():
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        aff = len(os.sched_getaffinity(0))
    except AttributeError:
        aff = os.cpu_count()
    return model, os.cpu_count(), aff


def cpu_baseline(workload, layers, head, target_s=15.0):
    """The fp64 oracle (as it stands) timed on the host on a bounded sample of
    the same workload: the full fwd + bwd of the first decoder layer's linears
    over their first Ts tokens (Ts chosen so the sample takes about
    `target_s`), plus the frozen head's dx on 64 sampled rows when the
    workload has one.  Every oracle function is linear in the token count, so
    the whole step is extrapolated as layers x (T / Ts) x the layer sample plus
    (T / 64) x the head sample, and labelled as such.  A 1-thread time of the
    first linear over a shorter token sample is reported beside it."""
    import oracle
    from workloads import sample_rows

    orc = oracle.load()
    threads = orc.threads()
    T = workload.tokens
    first = layers[:len(workload.linears)]
    cpu = [{k: getattr(L, k).cpu() for k in ("x", "W", "A", "B", "dy")} for L in first]

    def run_linear(i, Ts):
        L, c = first[i], cpu[i]
        s = L.lin.scale
        x, dy = c["x"][:Ts], c["dy"][:Ts]
        U = orc.u(x, c["A"])
        orc.y(x, c["W"], U, c["B"], s)
        _, dU = orc.grad_u(dy, c["B"], s)
        orc.dx(dy, c["W"], dU, c["A"])
        orc.da(dU, x)
        orc.db(dy, U, s)

    def run_layer(Ts):
        t0 = time.perf_counter()
        for i in range(len(first)):
            run_linear(i, Ts)
        return time.perf_counter() - t0

    def layer_flops(Ts):
        return sum(4.0 * Ts * L.lin.d_in * L.lin.d_out + 6.0 * Ts * L.lin.rank * (L.lin.d_in + L.lin.d_out)
                   for L in first)

    head_s, head_flops = 0.0, 0.0
    if head is not None:
        rows = sample_rows(T, 64)
        dyh, Wh = head[0].cpu()[rows], head[1].cpu()
        t0 = time.perf_counter()
        orc.frozen_dx(dyh, Wh)
        head_s = time.perf_counter() - t0
        head_flops = 2.0 * len(rows) * Wh.shape[0] * Wh.shape[1]
    run_layer(min(T, 16))  # warm-up: the thread pool and the caches
    Ts = min(T, 96)
    t = run_layer(Ts)
    budget = max(1.0, target_s - head_s)
    Ts = int(max(16, min(T, Ts * budget / max(t, 1e-3))))
    t = run_layer(Ts)
    value = (layer_flops(Ts) + head_flops) / (t + head_s) / 1e12
    step_s = workload.layers * t * T / Ts + (head_s * T / len(rows) if head is not None else 0.0)
    # 1 thread, first linear, shorter token sample
    orc.set_threads(1)
    try:
        L0 = first[0].lin
        # about 2 s at one thread: the layer sample's rate divided by the threads
        f0 = 4.0 * L0.d_in * L0.d_out + 6.0 * L0.rank * (L0.d_in + L0.d_out)
        T1 = max(8, min(T, int(2.0 * layer_flops(Ts) / max(t, 1e-3) / threads / f0)))
        t0 = time.perf_counter()
        run_linear(0, T1)
        t1 = time.perf_counter() - t0
    finally:
        orc.set_threads(threads)
    f1 = 4.0 * T1 * L0.d_in * L0.d_out + 6.0 * T1 * L0.rank * (L0.d_in + L0.d_out)
    model, ncpu, aff = cpu_info()
    what = (f"full fwd+bwd of the first layer's {len(first)} linear(s) over their first {Ts} of {T} tokens "
            f"({t:.1f} s)")
    if head is not None:
        what += f", plus the frozen head dx on 64 sampled rows ({head_s:.1f} s)"
    return {"value": value, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": what + "; fp64 C loops (OpenMP)",
            "cpu_model": model, "nproc": ncpu, "affinity_cpus": aff,
            "extrapolated_step_s": round(step_s, 1),
            "extrapolated_note": f"extrapolated: {workload.layers} layer(s) x T/{Ts} x the layer sample"
                                 + (" + T/64 x the head sample" if head is not None else "")
                                 + " (every oracle sum is linear in the token count)",
            "one_thread": {"value": f1 / t1 / 1e12, "unit": "TFLOP/s",
                           "sample": f"{L0.name} ({L0.d_in}->{L0.d_out}, r={L0.rank}) over {T1} tokens, "
                                     f"{t1:.1f} s"}}


def bench_workload(w, dev, steps, warmup, flush):
    """Warm and cold per-step times of one workload (the breakdown beside the
    headline): median / p10 / p90 and TFLOP/s on the median."""
    layers, head, ws, ws_bytes = build(w, dev)
    fn = lambda: step(layers, head, ws)  # noqa: E731
    for _ in range(warmup):
        fn()
    _, warm = event_steps(fn, steps)
    _, cold = event_steps(fn, steps, flush=flush)
    flops = w.flops_per_step()
    wm, cm = percentiles(warm), percentiles(cold)
    out = {"warm": wm, "cold": cm,
           "tflops_warm_median": round(flops / (wm["median_ms"] * 1e-3) / 1e12, 2),
           "tflops_cold_median": round(flops / (cm["median_ms"] * 1e-3) / 1e12, 2),
           "frac_bf16_peak_warm": round(flops / (wm["median_ms"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
           "steps": steps, "workspace_bytes": int(ws_bytes)}
    pk = per_kernel_ms(fn, steps)
    out["kernels"] = kernel_table(w, pk, steps)
    del layers, head, ws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama_stack", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-workload breakdown of the smaller workloads")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache pass")
    ap.add_argument("--no-topk", action="store_true",
                    help="skip the secondary measurement of the top-k similarity table build")
    ap.add_argument("--no-ckpt", action="store_true",
                    help="skip the secondary measurement of the checkpointed chain")
    ap.add_argument("--no-head", action="store_true",
                    help="skip the secondary measurement of the reduced-vocabulary LM head")
    ap.add_argument("--no-quant", action="store_true",
                    help="skip the secondary measurement with the quantized frozen base")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the steps, copy a buffer of this many MiB (device to device) so a "
                         "counter run can calibrate FETCH_SIZE / WRITE_SIZE against known bytes")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): the LoRA hot path is "
              "measured on one MI355X; multi-GPU data parallelism is a design note, not a "
              "measured configuration.", file=sys.stderr)
        sys.exit(2)

    w = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    log(f"[bench] workload {w.key}: {w.description}")
    layers, head, ws, ws_bytes = build(w, dev)
    torch.cuda.synchronize()
    base_mem = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    fn = lambda: step(layers, head, ws)  # noqa: E731

    for _ in range(args.warmup):
        fn()
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup} done")

    # Timed region: exactly K steps between two synchronisations, an event
    # between consecutive steps (per-step spread).
    total_ms, per = event_steps(fn, args.steps)
    ms = total_ms / args.steps
    log(f"[bench] {args.steps} steps: {ms:.4f} ms/step")
    extra_peak = torch.cuda.max_memory_allocated() - base_mem
    total_peak = torch.cuda.max_memory_allocated()
    if lm.handover_giveups():
        raise RuntimeError("a fused hand-over wait gave up during the timed steps")

    timing = {"warm": percentiles(per)}
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    if not args.no_cold:
        _, cold = event_steps(fn, args.steps, flush=flush)
        timing["cold"] = percentiles(cold)
        log(f"[bench] cold-cache median {timing['cold']['median_ms']:.4f} ms/step")

    # Same steps again with the library's HIP-event hook around every kernel.
    per_kernel = per_kernel_ms(fn, args.steps)
    kernels = kernel_table(w, per_kernel, args.steps)
    gemms = {k: v for k, v in kernels.items() if v.get("bound") == "mfma"}
    dom = max(gemms, key=lambda k: gemms[k]["ms_per_step"])
    kd = kernels[dom]
    traffic = stored_traffic(w.key).get(dom)
    roofline = {"bound": "mfma", "achieved": kd["achieved"], "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": kd["frac"], "traffic": traffic, "kernel": dom,
                "avg_launch_us": kd["avg_launch_us"], "flops_per_launch": kd["flops_per_launch"]}
    log("[bench] per-kernel: " + ", ".join(f"{k}={v['ms_per_step']:.3f} ms ({v.get('frac')})"
                                           for k, v in kernels.items()))

    flops = w.flops_per_step()
    value = flops / (ms * 1e-3) / 1e12
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.key, "tokens": w.tokens,
                   "linears": [[l.name, l.d_in, l.d_out, l.rank, l.alpha] for l in w.linears],
                   "layers": w.layers,
                   "head": None if w.head is None else [w.head.d_in, w.head.d_out],
                   "parallelism": "single GPU"},
        "frac_bf16_peak": round(value / PEAK_BF16_TFLOPS, 4),
        "timing": timing,
        "timing_note": "value and ms_per_step: K back-to-back steps (warm: a step's inputs may sit "
                       "in the 256 MB last-level cache from the step before); cold: each step after "
                       "a 512 MiB write that evicts that cache",
        "peak_workspace_bytes": int(ws_bytes),
        "peak_extra_device_bytes_during_steps": int(extra_peak),
        "total_device_bytes_peak": int(total_peak),
        "frozen_weight_bytes": int(w.frozen_weight_bytes()),
        "roofline": roofline,
        "kernels": kernels,
    }
    if not args.no_quant:
        # Quantized frozen base (INT4 linears, INT8 head) dequantized inside the
        # GEMMs: same workload, same flop count, weights read as codes.
        qs, qh = build_quant(layers, head, w, dev)
        fq = lambda: step_quant(layers, head, ws, qs, qh)  # noqa: E731
        msq = time_steps(fq, args.steps, args.warmup)
        pk = per_kernel_ms(fq, args.steps)
        wbytes = sum(q["codes"].numel() + 2 * q["scale"].numel() * 4 for q in qs)
        if qh is not None:
            wbytes += qh["codes"].numel() + 2 * qh["scale"].numel() * 4
        out["quantized_base"] = {
            "weights": "INT4 codes, groups of 128, fp32 scale and offset"
                       + ("; head INT8" if qh is not None else ""),
            "ms_per_step": round(msq, 5), "value": round(flops / (msq * 1e-3) / 1e12, 2),
            "unit": "TFLOP/s", "frozen_weight_bytes": int(wbytes),
            "kernels_ms_per_step": {k: round(v[0] / args.steps, 5) for k, v in pk.items()}}
        log(f"[bench] quantized base: {msq:.4f} ms/step")
        del qs, qh
    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle) ...")
        cpu = cpu_baseline(w, layers, head)
    del layers, head, ws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if not args.no_configs:
        cfgs = {}
        for key in ORDER:
            if key == w.key:
                continue
            n = {"single_256": 200, "llama_q_proj": 200}.get(key, 50)
            cfgs[key] = bench_workload(WORKLOADS[key], dev, n, 5, flush)
            log(f"[bench] {key}: {cfgs[key]['warm']['median_ms']:.4f} ms/step warm, "
                f"{cfgs[key]['cold']['median_ms']:.4f} cold")
        out["configs"] = cfgs
    if not args.no_topk:
        out["topk_table"] = bench_topk(dev)
        log(f"[bench] top-k table: {out['topk_table']}")
    if not args.no_ckpt:
        out["checkpointed_chain"] = bench_ckpt(dev)
        log(f"[bench] checkpointed chain: {out['checkpointed_chain']}")
    if not args.no_head:
        out["lm_head_reduced"] = bench_lm_head(dev)
        log(f"[bench] lm head: {out['lm_head_reduced']}")
    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["calib_copy_bytes"] = n * 4
    if lm.handover_giveups():
        raise RuntimeError("a fused hand-over wait gave up during the benchmark")
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
