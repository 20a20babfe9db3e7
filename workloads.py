"""Seeded synthetic workloads for the LoRA linear hot path.

This module holds shapes and random-number recipes only -- none of the
method's arithmetic.  The tests, the smoke check and the benchmark draw their
inputs here; both the oracle and the HIP path then consume the very same
bytes.

Recipe (one LoRA linear, d_in = K, d_out = N):
    x  ~ N(0, 1)             [T, K]
    W  ~ N(0, 0.02)          [N, K]   (frozen base weight; 0.02 is a std. dev.)
    A  ~ U(-1/sqrt(K), 1/sqrt(K))  [r, K]
    B  ~ N(0, 0.02)          [N, r]
    dy ~ N(0, 1)             [T, N]   (synthetic upstream gradient)
drawn in fp32 in that order from one seeded torch generator, then rounded to
the compute dtype with round-to-nearest-even.  Every LoRA linear uses
scale s = alpha / r.

The layer shapes stand in for the paper's Llama-3.2-3B and Qwen-2.5-3B
fine-tuning runs (LoRA r=16, alpha=16 in its hyperparameter table; the
vocabulary sizes of its model-configuration appendix); the token counts span
the context lengths of its peak-memory tables.  Real text (the XSum / SQuAD
runs) is replaced by these Gaussian stand-ins.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

LLAMA32_3B_VOCAB = 128256  # vocabulary size stated in the paper's model-configuration appendix


@dataclass(frozen=True)
class Linear:
    name: str
    d_in: int
    d_out: int
    rank: int          # 0 = frozen linear, input gradient only
    alpha: float

    @property
    def scale(self) -> float:
        return self.alpha / self.rank if self.rank else 0.0


@dataclass(frozen=True)
class Workload:
    key: str
    description: str
    tokens: int
    linears: tuple = field(default_factory=tuple)
    layers: int = 1                       # the linears repeat this many times
    head: Linear | None = None            # optional frozen rank-0 LM head

    def flops_per_step(self) -> float:
        """Algorithmic flops of one fwd+bwd over every linear: 4TKN + 6Tr(K+N)
        per LoRA linear (fwd x W^T, bwd dy W, plus the rank-r products), 2TKN for
        a frozen dx-only linear."""
        T = self.tokens
        f = 0.0
        for lin in self.linears:
            K, N, r = lin.d_in, lin.d_out, lin.rank
            f += 4.0 * T * K * N + 6.0 * T * r * (K + N)
        f *= self.layers
        if self.head is not None:
            f += 2.0 * T * self.head.d_in * self.head.d_out
        return f

    def frozen_weight_bytes(self, elem: int = 2) -> int:
        b = sum(l.d_in * l.d_out for l in self.linears) * self.layers
        if self.head is not None:
            b += self.head.d_in * self.head.d_out
        return b * elem


def _llama_layer(r: int, alpha: float):
    h, kv, mlp = 3072, 1024, 8192
    return (Linear("q_proj", h, h, r, alpha), Linear("k_proj", h, kv, r, alpha),
            Linear("v_proj", h, kv, r, alpha), Linear("o_proj", h, h, r, alpha),
            Linear("gate_proj", h, mlp, r, alpha), Linear("up_proj", h, mlp, r, alpha),
            Linear("down_proj", mlp, h, r, alpha))


WORKLOADS = {
    "single_256": Workload(
        "single_256", "single LoRA linear 256->256, T=128, r=8, alpha=16", 128,
        (Linear("linear", 256, 256, 8, 16.0),)),
    "llama_q_proj": Workload(
        "llama_q_proj", "Llama-3.2-3B-shaped q_proj 3072->3072, T=1024, r=16, alpha=32", 1024,
        (Linear("q_proj", 3072, 3072, 16, 32.0),)),
    "llama_mlp": Workload(
        "llama_mlp", "Llama-3.2-3B-shaped MLP (gate/up 3072->8192, down 8192->3072), T=2048, r=16, alpha=32",
        2048, (Linear("gate_proj", 3072, 8192, 16, 32.0), Linear("up_proj", 3072, 8192, 16, 32.0),
               Linear("down_proj", 8192, 3072, 16, 32.0))),
    "qwen_layer": Workload(
        "qwen_layer", "Qwen-2.5-3B-shaped decoder layer (q/o 2048^2, k/v 2048->256, MLP 2048<->11008), "
                      "T=2048, r=8, alpha=16", 2048,
        (Linear("q_proj", 2048, 2048, 8, 16.0), Linear("k_proj", 2048, 256, 8, 16.0),
         Linear("v_proj", 2048, 256, 8, 16.0), Linear("o_proj", 2048, 2048, 8, 16.0),
         Linear("gate_proj", 2048, 11008, 8, 16.0), Linear("up_proj", 2048, 11008, 8, 16.0),
         Linear("down_proj", 11008, 2048, 8, 16.0))),
    "llama_stack": Workload(
        "llama_stack", "28-layer Llama-3.2-3B-shaped stack of LoRA linears, T=4096, r=32, alpha=64, "
                       "plus a frozen rank-0 LM head 3072->128256 (dx only)", 4096,
        _llama_layer(32, 64.0), layers=28, head=Linear("lm_head", 3072, LLAMA32_3B_VOCAB, 0, 0.0)),
}

# Ordered as the five workloads of the benchmark spec (small case first).
ORDER = ["single_256", "llama_q_proj", "llama_mlp", "qwen_layer", "llama_stack"]


def linear_seed(base_seed: int, layer: int, index: int) -> int:
    """Seed of linear `index` (0..6) in decoder layer `layer`: base + 7*layer + index."""
    return base_seed + 7 * layer + index


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def lora_inputs(T: int, d_in: int, d_out: int, r: int, seed: int = 0,
                dtype=torch.bfloat16, device="cpu") -> dict:
    """Draw x, W, A, B, dy (in that order) for one LoRA linear; see module doc."""
    g = _gen(seed, device)
    f32 = torch.float32
    x = torch.randn(T, d_in, generator=g, device=device, dtype=f32)
    W = torch.randn(d_out, d_in, generator=g, device=device, dtype=f32) * 0.02
    bound = 1.0 / (d_in ** 0.5)
    A = (torch.rand(r, d_in, generator=g, device=device, dtype=f32) * 2.0 - 1.0) * bound
    B = torch.randn(d_out, r, generator=g, device=device, dtype=f32) * 0.02
    dy = torch.randn(T, d_out, generator=g, device=device, dtype=f32)
    return {k: v.to(dtype).contiguous() for k, v in
            (("x", x), ("W", W), ("A", A), ("B", B), ("dy", dy))}


def frozen_inputs(T: int, d_in: int, d_out: int, seed: int = 0,
                  dtype=torch.bfloat16, device="cpu") -> dict:
    """Draw dy ~ N(0,1) [T, d_out] and W ~ N(0, 0.02) [d_out, d_in] for a rank-0 frozen linear."""
    g = _gen(seed, device)
    f32 = torch.float32
    W = torch.randn(d_out, d_in, generator=g, device=device, dtype=f32) * 0.02
    dy = torch.randn(T, d_out, generator=g, device=device, dtype=f32)
    return {"W": W.to(dtype).contiguous(), "dy": dy.to(dtype).contiguous()}


def quant_weight(d_out: int, d_in: int, bits: int = 4, group: int = 128, seed: int = 0,
                 device="cpu") -> dict:
    """A quantized frozen weight in the layout of the library's quantized entry
    points: codes ~ U{0 .. 2^bits - 1} packed along d_in (two 4-bit codes per
    byte, even input in the low nibble), and per (row, group) an fp32 scale
    ~ 0.02 * sqrt(12) / 2^bits * U(0.5, 1.5) and an fp32 offset centring the
    codes' range near zero, so that the weights spread like the N(0, 0.02)
    bf16 weights of lora_inputs.  Drawn in that order (codes, scale factor,
    offset jitter; scales and offsets row by row) from one seeded generator.
    scale and offset are stored group-major, [d_in / group][d_out] (their
    transposes are the [row][group] arrays the oracle's dequant takes)."""
    g = _gen(seed, device)
    levels = 1 << bits
    q = torch.randint(0, levels, (d_out, d_in), generator=g, device=device, dtype=torch.int32)
    if bits == 4:
        codes = (q[:, 0::2] | (q[:, 1::2] << 4)).to(torch.uint8)
    else:
        codes = q.to(torch.uint8)
    ng = d_in // group
    step = 0.02 * (12.0 ** 0.5) / levels
    scale = step * (0.5 + torch.rand(d_out, ng, generator=g, device=device))
    jitter = 0.25 * (torch.rand(d_out, ng, generator=g, device=device) - 0.5)
    offset = -scale * ((levels - 1) / 2.0 + jitter)
    return {"codes": codes.contiguous(), "scale": scale.float().t().contiguous(),
            "offset": offset.float().t().contiguous(), "bits": bits}


def head_inputs(T: int, V: int, D: int, ktab: int, trainable: float = 0.3, clusters: int = 64,
                spread: int = 32, seed: int = 0, device="cpu") -> dict:
    """Synthetic stand-ins for the frozen LM head's inputs:
      h ~ N(0, 1) [T, D] and W ~ N(0, 0.02) [V, D] (bf16), drawn in that order;
      targets y [T]: `clusters` centres ~ U{0..V-1}, each target a centre plus
      U{-spread..spread} (mod V), so that the targets share neighbourhoods as
      the tokens of one text do;
      table [V, ktab] int32: row v lists v, v+1, v-1, v+2, v-2, ... (mod V) --
      a stand-in for the similarity table in which the nearest tokens of v are
      its index neighbours (its first entry is v itself);
      rows: the trainable positions, the last `trainable` fraction of the
      sequence (the response after a prompt).
    All int32 except h, W."""
    g = _gen(seed, device)
    f32 = torch.float32
    h = torch.randn(T, D, generator=g, device=device, dtype=f32)
    W = torch.randn(V, D, generator=g, device=device, dtype=f32) * 0.02
    centres = torch.randint(0, V, (clusters,), generator=g, device=device)
    pick = torch.randint(0, clusters, (T,), generator=g, device=device)
    off = torch.randint(-spread, spread + 1, (T,), generator=g, device=device)
    y = (centres[pick] + off) % V
    c = torch.arange(ktab, device=device)
    step = (c + 1) // 2 * torch.where(c % 2 == 1, 1, -1)
    table = (torch.arange(V, device=device)[:, None] + step[None, :]) % V
    n_train = max(1, int(round(T * trainable)))
    rows = torch.arange(T - n_train, T, device=device)
    return {"h": h.to(torch.bfloat16).contiguous(), "W": W.to(torch.bfloat16).contiguous(),
            "targets": y.to(torch.int32).contiguous(), "table": table.to(torch.int32).contiguous(),
            "rows": rows.to(torch.int32).contiguous()}


def sample_rows(T: int, n: int = 64, seed: int = 1234) -> list:
    """Deterministic sorted sample of row indices, always including the first and
    last rows (the ragged-tail tile), of size min(n, T)."""
    if T <= n:
        return list(range(T))
    g = torch.Generator().manual_seed(seed)
    mid = torch.randperm(T - 2, generator=g)[: n - 2] + 1
    return sorted({0, T - 1, *mid.tolist()})
