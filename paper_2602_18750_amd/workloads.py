"""Seeded synthetic decode-step inputs for the five benchmark workloads.

This module only draws random numbers: it holds none of the method's
arithmetic, and it is the single piece of code that both the GPU path's
tests/benchmark and the CPU oracle consume.

There is no public dataset behind these workloads: the paper's models,
LongBench / PG-19 text and LM-eval tasks are replaced by random tensors with
the head layout of the architectures the workloads are named after
(Qwen-7B: 32 MHA heads x 128; Llama-3-8B: 32 query / 8 KV heads x 128).

Recipe (per layer): ``torch.Generator(device).manual_seed(seed)``; draw K,
then V, then the auxiliary tensors (heavy-hitter positions or per-channel
outlier scales), then the queries for steps 0..T-1, every draw with
``torch.randn`` in float32 and a final cast to fp16/bf16 (round to nearest
even).  Seed = 0 for the 4K single-layer MHA case and ``1000*id + layer``
otherwise.  Layouts: K, V ``[B, Hkv, n, D]`` contiguous; q ``[T, B, Hq, D]``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import torch

__all__ = ["Workload", "WORKLOADS", "sweep_workloads", "LayerInputs", "make_layer",
           "make_random", "layer_seed", "budget_tokens"]


@dataclasses.dataclass(frozen=True)
class Workload:
    id: int
    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    n_tokens: int
    dtype: str            # "fp16" | "bf16"
    budget: float         # alpha, fraction of tokens kept
    steps: int            # decode steps
    layers: int
    keys: str             # "normal" | "heavy" | "outlier"
    queries: str          # "iid" | "ar1"

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    @property
    def k_sel(self) -> int:
        return budget_tokens(self.n_tokens, self.budget)

    @property
    def torch_dtype(self):
        return torch.float16 if self.dtype == "fp16" else torch.bfloat16


def budget_tokens(n: int, alpha: float) -> int:
    """floor(alpha * n) clamped to [1, n]; e.g. 20% of 4096 -> 819."""
    return max(1, min(n, int(math.floor(alpha * n + 1e-9))))


WORKLOADS = {
    1: Workload(1, "mha32-b1-n4096-fp16", 1, 32, 32, 128, 4096, "fp16", 0.20, 1, 1,
                "normal", "iid"),
    2: Workload(2, "qwen7b-mha32-b8-n4096-fp16-heavy", 8, 32, 32, 128, 4096, "fp16", 0.20, 1, 32,
                "heavy", "iid"),
    3: Workload(3, "llama3-8b-gqa32x8-b1-n32768-bf16-outlier", 1, 32, 8, 128, 32768, "bf16", 0.10,
                64, 32, "outlier", "iid"),
    4: Workload(4, "gqa32x8-b4-n131072-bf16-ar1", 4, 32, 8, 128, 131072, "bf16", 0.05, 16, 1,
                "normal", "ar1"),
}


def sweep_workloads() -> List[Workload]:
    """The 27-cell throughput sweep: B x n x alpha, GQA 32/8, bf16, one step."""
    cells = []
    for b in (1, 8, 32):
        for n in (8192, 32768, 65536):
            for a in (0.05, 0.10, 0.20):
                cells.append(Workload(5, "sweep-b%d-n%d-a%d" % (b, n, round(a * 100)), b, 32, 8, 128,
                                      n, "bf16", a, 1, 1, "normal", "iid"))
    return cells


def layer_seed(w: Workload, layer: int) -> int:
    return 0 if w.id == 1 else 1000 * w.id + layer


@dataclasses.dataclass
class LayerInputs:
    q: torch.Tensor                 # [T, B, Hq, D]
    k: torch.Tensor                 # [B, Hkv, n, D]
    v: torch.Tensor                 # [B, Hkv, n, D]
    heavy: Optional[torch.Tensor]   # [B, n_heavy] positions with 4x keys, or None


HEAVY_FRACTION = 0.05
HEAVY_GAIN = 4.0
AR_RHO = 0.95


def make_layer(w: Workload, layer: int = 0, device="cpu", seed: Optional[int] = None) -> LayerInputs:
    """Draw one layer's K, V and the queries of all its decode steps."""
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(layer_seed(w, layer) if seed is None else seed)
    B, Hq, Hkv, D, n, T = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.n_tokens, w.steps
    k = torch.randn((B, Hkv, n, D), generator=g, device=dev, dtype=torch.float32)
    v = torch.randn((B, Hkv, n, D), generator=g, device=dev, dtype=torch.float32)
    heavy = None
    if w.keys == "heavy":
        nh = int(math.floor(HEAVY_FRACTION * n))
        heavy = torch.stack([torch.randperm(n, generator=g, device=dev)[:nh] for _ in range(B)])
        for b in range(B):
            k[b, :, heavy[b], :] *= HEAVY_GAIN
    elif w.keys == "outlier":
        # per (KV head, channel) scale c = exp(N(0,1)), i.e. LogNormal(0, 1)
        c = torch.exp(torch.randn((Hkv, D), generator=g, device=dev, dtype=torch.float32))
        k *= c[None, :, None, :]
    elif w.keys != "normal":
        raise ValueError(w.keys)
    eps = torch.randn((T, B, Hq, D), generator=g, device=dev, dtype=torch.float32)
    if w.queries == "ar1":
        q = torch.empty_like(eps)
        q[0] = eps[0]
        s = math.sqrt(1.0 - AR_RHO * AR_RHO)
        for t in range(1, T):
            q[t] = AR_RHO * q[t - 1] + s * eps[t]
    elif w.queries == "iid":
        q = eps
    else:
        raise ValueError(w.queries)
    dt = w.torch_dtype
    return LayerInputs(q=q.to(dt), k=k.to(dt), v=v.to(dt), heavy=heavy)


def make_random(B, Hq, Hkv, D, n, dtype="fp16", steps=1, seed=0, device="cpu",
                keys="normal", queries="iid") -> LayerInputs:
    """Same recipe at an arbitrary shape (tests: ragged sizes, tiny cases)."""
    w = Workload(0, "custom", B, Hq, Hkv, D, n, dtype, 0.1, steps, 1, keys, queries)
    return make_layer(w, 0, device=device, seed=seed)
