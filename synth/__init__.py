"""Seeded synthetic inputs shaped like the paper's workloads.

This module is shared by the parity tests, the benchmark and the oracle's
callers.  It holds none of the method's arithmetic (no inclusion
probabilities, no sampling, no Hajek weights, no certificate): it only draws
caches, queries and importance scores.

Recipe (stated once, used everywhere):
  * K, V, q ~ N(0, 1), rounded to bf16 (round to nearest even).
  * Heavy hitters: an independent Bernoulli(2%) per (unit, token) scales that
    token's key by 4 (exact in bf16).
  * Importance scores ("window" recipe): for each unit, 32 window queries
    q_w ~ N(0, 1); score_i = sum_w softmax_i(q_w . k_i / sqrt(d)) over the
    unit's full cache, in fp32.  This stands in for the accumulated-attention
    importance the paper feeds its sampler (App. B, harness); the paper's
    models and prompts are not available, so only the shapes are reproduced.
  * Long-context recipe ("pareto"): score_i = (1 - U)^(-1/alpha), alpha = 1.5
    (Pareto I with x_m = 1), independent of the keys -- the poorly aligned
    score case the paper discusses under Assumption 2.

All tensors are produced with torch on the requested device from a seeded
torch.Generator, so the same seed gives the same inputs on a given device.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional, Sequence

import torch

HEAD_DIM = 128


@dataclass(frozen=True)
class Workload:
    """A workload by shape: units = layers x batch x KV heads (one cache each)."""

    name: str
    layers: int
    batch: int
    kv_heads: int
    group: int  # query heads per KV head
    context: int
    budgets: Sequence[float]
    pi_min: float = 0.01
    n_sink: int = 4
    n_recent: int = 64
    decode_steps: int = 1
    scores: str = "window"  # "window" | "pareto"
    head_dim: int = HEAD_DIM
    description: str = ""

    @property
    def units(self) -> int:
        return self.layers * self.batch * self.kv_heads


WORKLOADS = {
    "single_layer_4k": Workload(
        "single_layer_4k", layers=1, batch=1, kv_heads=8, group=1, context=4096, budgets=(0.10,),
        description="1 layer, batch 1, 8 KV heads = 8 query heads, context 4096, 10% budget"),
    "qwen7b_6k": Workload(
        "qwen7b_6k", layers=28, batch=16, kv_heads=4, group=7, context=6144,
        budgets=(0.10, 0.25, 0.50),
        description="Qwen2.5-7B-shaped: 28 layers, 28 query / 4 KV heads, batch 16, context 6144"),
    "llama8b_16k": Workload(
        "llama8b_16k", layers=32, batch=32, kv_heads=8, group=4, context=16384, budgets=(0.25,),
        decode_steps=64,
        description="Llama-3-8B-shaped: 32 layers, 32 query / 8 KV heads, batch 32, context 16384"),
    "long_128k": Workload(
        "long_128k", layers=32, batch=4, kv_heads=8, group=4, context=131072, budgets=(0.10,),
        pi_min=0.005, decode_steps=128, scores="pareto",
        description="long context: 32 layers, 32 query / 8 KV heads, batch 4, context 131072"),
}

REPLAY_BUDGETS = (0.05, 0.10, 0.15, 0.25, 0.50)
REPLAY_CONTEXTS = (2048, 6144, 16384)
REPLAY_CELLS = 12096
REPLAY_KV_HEADS = 8


def replay_cell(c: int):
    """Cell c of the replay grid -> (budget, context, data stream, layer tag)."""
    budget = REPLAY_BUDGETS[c % 5]
    context = REPLAY_CONTEXTS[(c // 5) % 3]
    stream = c // 15
    layer = (c // 15) % 28
    return budget, context, stream, layer


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def seq_offsets(lengths: Sequence[int], device="cpu") -> torch.Tensor:
    off = [0]
    for n in lengths:
        off.append(off[-1] + int(n))
    return torch.tensor(off, dtype=torch.int64, device=device)


def normal_bf16(shape, gen: torch.Generator, device) -> torch.Tensor:
    return torch.randn(shape, generator=gen, device=device, dtype=torch.float32).to(torch.bfloat16)


def make_cache(lengths: Sequence[int], seed: int = 0, device="cpu", d: int = HEAD_DIM,
               hh_frac: float = 0.02, hh_scale: float = 4.0, chunk_rows: int = 1 << 24):
    """K, V bf16 [sum(lengths), d] (unit u owns rows seq_off[u]:seq_off[u+1]) and seq_off."""
    rows = int(sum(int(n) for n in lengths))
    g = _gen(seed, device)
    K = torch.empty((rows, d), dtype=torch.bfloat16, device=device)
    V = torch.empty((rows, d), dtype=torch.bfloat16, device=device)
    for r0 in range(0, rows, chunk_rows):
        r1 = min(rows, r0 + chunk_rows)
        k = torch.randn((r1 - r0, d), generator=g, device=device, dtype=torch.float32)
        hh = torch.rand((r1 - r0, 1), generator=g, device=device) < hh_frac
        k = torch.where(hh, k * hh_scale, k)
        K[r0:r1] = k.to(torch.bfloat16)
        V[r0:r1] = torch.randn((r1 - r0, d), generator=g, device=device,
                               dtype=torch.float32).to(torch.bfloat16)
    return K, V, seq_offsets(lengths, device)


def make_queries(units: int, group: int, seed: int = 1, device="cpu", d: int = HEAD_DIM):
    """Decode queries q bf16 [units, group, d]."""
    return normal_bf16((units, group, d), _gen(seed, device), device)


def window_scores(K: torch.Tensor, seq_off: torch.Tensor, n_window: int = 32, seed: int = 2,
                  max_elems: int = 1 << 27) -> torch.Tensor:
    """Importance = attention mass summed over n_window random queries, per unit (fp32)."""
    device = K.device
    d = K.shape[1]
    g = _gen(seed, device)
    off = seq_off.tolist()
    U = len(off) - 1
    out = torch.empty((K.shape[0],), dtype=torch.float32, device=device)
    qw_all = torch.randn((U, n_window, d), generator=g, device=device, dtype=torch.float32)
    scale = 1.0 / math.sqrt(d)
    # Uniform-length runs of units are batched; ragged units go one at a time.
    u = 0
    while u < U:
        n = off[u + 1] - off[u]
        v = u + 1
        while v < U and off[v + 1] - off[v] == n and (v - u + 1) * n * n_window <= max_elems:
            v += 1
        if n > 0:
            k = K[off[u]:off[v]].view(v - u, n, d).to(torch.float32)
            qt = qw_all[u:v].transpose(1, 2).contiguous()  # [b, d, W]
            logits = torch.matmul(k, qt) * scale  # [b, n, W]
            p = torch.softmax(logits, dim=1)
            out[off[u]:off[v]] = p.sum(dim=2).reshape(-1)
        u = v
    return out


def pareto_scores(rows: int, alpha: float = 1.5, seed: int = 2, device="cpu") -> torch.Tensor:
    u = torch.rand((rows,), generator=_gen(seed, device), device=device, dtype=torch.float64)
    return torch.pow(1.0 - u, -1.0 / alpha).to(torch.float32)


def make_workload_inputs(wl: Workload, units: Optional[int] = None, seed: int = 0, device="cpu"):
    """Full inputs for `units` units of a workload (defaults to all of them)."""
    U = wl.units if units is None else int(units)
    K, V, seq_off = make_cache([wl.context] * U, seed=seed, device=device, d=wl.head_dim)
    if wl.scores == "pareto":
        scores = pareto_scores(K.shape[0], seed=seed + 2, device=device)
    else:
        scores = window_scores(K, seq_off, seed=seed + 2)
    q = make_queries(U, wl.group, seed=seed + 1, device=device, d=wl.head_dim)
    return {"K": K, "V": V, "seq_off": seq_off, "scores": scores, "q": q}


def bf16_bits(t: torch.Tensor):
    """bf16 tensor -> numpy uint16 bit patterns (host copy)."""
    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view("uint16")
