"""Seeded synthetic workloads with the shapes of the paper's evaluation models.

Inputs only: this module holds none of the selection arithmetic. It draws the
window queries, keys and values, the chosen-head mask and the normalised layer
errors, and plants structure the selection should find:

  * queries, keys, values ~ N(0, 1) in fp32, rounded once to the workload dtype
    (round to nearest even);
  * "sink" keys at positions 0..sinks-1 and n_spans non-overlapping spans of
    span_len keys, each shifted by delta_g = 3 * sqrt(d) * qbar_g / |qbar_g|^2,
    where qbar_g is the mean of group g's chosen window queries, so the mean
    scaled logit of the chosen rows on a planted key rises by 3;
  * the head mask chooses n heads per group without replacement, n drawn from
    the workload's choices;
  * normalised layer errors ~ Dirichlet(1, ..., 1) for Algorithm 1.

Shapes: GQA attention layers like Llama-3.1-8B / Mistral-7B (32 query heads,
8 KV heads, head_dim 128, 32 layers) and Qwen2.5-7B (28 query heads, 4 KV
heads, 28 layers). The paper's LongBench / Needle-in-a-Haystack prompts and the
models' real activations are not available; these draws stand in for them.

Seeds: workload c uses base seed 1000*c; layer l of it uses 1000*c + l + 1.
Random numbers come from torch generators on the target device (so large
workloads are drawn on the GPU) and numpy PCG64 for the small host draws.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    index: int                     # base seed = 1000 * index
    n_layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    seq_lens: Tuple[int, ...]      # one entry per prompt of the batch
    window: int
    n_sel_choices: Tuple[int, ...]
    pool: int                      # 0 average, 1 max
    pool_kernel: int
    dtype: torch.dtype
    sinks: int
    n_spans: int
    span_len: int
    # budgets: a fixed per-layer budget, or Algorithm 1 parameters
    budget: Optional[int] = None
    avg_budget: Optional[int] = None      # B_total = n_layers * avg_budget
    budget_ratio: Optional[float] = None  # B_total = n_layers * round(ratio * L)
    m: int = 32
    description: str = ""


WORKLOADS: Dict[str, Workload] = {w.name: w for w in [
    Workload("tiny-fp32", 1, 1, 8, 2, 64, (1024,), 16, (1,), 0, 7, torch.float32,
             4, 1, 16, budget=128,
             description="1 layer, 8 q / 2 kv heads, d=64, L=1024, fp32, w=16, 1 head/group, "
                         "avgpool 7, B=128"),
    Workload("llama8b-32k-layer", 2, 1, 32, 8, 128, (32768,), 32, (2,), 1, 7, torch.bfloat16,
             4, 8, 32, budget=2048,
             description="1 Llama-3.1-8B-shaped layer, L=32768, bf16, w=32, 2 heads/group, "
                         "maxpool 7, B=2048"),
    Workload("llama8b-32k-stack", 3, 32, 32, 8, 128, (32768,), 32, (1, 2), 1, 7, torch.bfloat16,
             4, 8, 32, avg_budget=512, m=32,
             description="32 Llama-3.1-8B-shaped layers, L=32768, bf16, w=32, 1-2 heads/group, "
                         "maxpool 7, Algorithm 1 budgets averaging 512"),
    Workload("llama8b-128k-stack", 4, 32, 32, 8, 128, (131072,), 64, (1, 2), 1, 7, torch.bfloat16,
             4, 64, 8, avg_budget=128, m=64,
             description="32 Llama-3.1-8B-shaped layers, L=131072, bf16, w=64, 1-2 heads/group, "
                         "maxpool 7, Algorithm 1 budgets averaging 128 (~0.1%)"),
    Workload("qwen7b-ragged-batch", 5, 28, 28, 4, 128, (8192, 24576, 65536, 98304), 32, (2,), 1, 7,
             torch.bfloat16, 4, 8, 32, budget_ratio=0.03, m=32,
             description="28 Qwen2.5-7B-shaped layers, 28 q / 4 kv heads, ragged batch "
                         "L={8192,24576,65536,98304}, bf16, w=32, 2 heads/group, maxpool 7, "
                         "Algorithm 1 budgets totalling 3% of each prompt"),
]}


def layer_seed(wl: Workload, layer: int) -> int:
    return 1000 * wl.index + layer + 1


def head_mask(wl: Workload, layer: int) -> np.ndarray:
    """uint8 [H]: n chosen heads per group, n from the workload's choices."""
    rng = np.random.default_rng(layer_seed(wl, layer))
    G = wl.num_q_heads // wl.num_kv_heads
    mask = np.zeros(wl.num_q_heads, dtype=np.uint8)
    for g in range(wl.num_kv_heads):
        n = int(rng.choice(wl.n_sel_choices))
        for t in rng.choice(G, size=n, replace=False):
            mask[g * G + int(t)] = 1
    return mask


def shared_head_mask(wl: Workload, layer: int, n_heads: int = 4) -> np.ndarray:
    """uint8 [H]: n_heads retrieval heads of the whole layer, drawn uniformly
    from all query heads (any groups, several may share one), the paper's
    layer-shared setting (its top-4 heads per layer)."""
    rng = np.random.default_rng([layer_seed(wl, layer), 4])
    mask = np.zeros(wl.num_q_heads, dtype=np.uint8)
    mask[rng.choice(wl.num_q_heads, size=n_heads, replace=False)] = 1
    return mask


def layer_errors(wl: Workload) -> np.ndarray:
    """Normalised per-layer errors ~ Dirichlet(1) (input to Algorithm 1)."""
    rng = np.random.default_rng(1000 * wl.index)
    return rng.dirichlet(np.ones(wl.n_layers))


def budget_params(wl: Workload, seq_len: int) -> Tuple[int, int, int]:
    """(B_total, m, M) for Algorithm 1 on one prompt; M = 3 * B_total / n_layers."""
    if wl.avg_budget is not None:
        total = wl.n_layers * wl.avg_budget
    elif wl.budget_ratio is not None:
        total = wl.n_layers * int(round(wl.budget_ratio * seq_len))
    else:
        total = wl.n_layers * wl.budget
    return total, wl.m, (3 * total) // wl.n_layers


def planted_positions(wl: Workload, layer: int, seq: int, seq_len: int) -> np.ndarray:
    """Sink positions plus non-overlapping span positions inside the prefix."""
    rng = np.random.default_rng([layer_seed(wl, layer), seq, 7])
    lo, hi = wl.sinks, seq_len - wl.window - wl.span_len
    n_slots = max((hi - lo) // wl.span_len, 0)
    n = min(wl.n_spans, n_slots)
    slots = np.sort(rng.choice(n_slots, size=n, replace=False)) if n else np.zeros(0, np.int64)
    pos = [np.arange(wl.sinks)]
    for s in slots:
        start = lo + int(s) * wl.span_len
        pos.append(np.arange(start, start + wl.span_len))
    return np.concatenate(pos).astype(np.int64)


@dataclass
class LayerInputs:
    q_win: List[torch.Tensor]            # per prompt [H, w, d]
    k: List[torch.Tensor]                # per prompt [n_kv, L, d]
    v: List[torch.Tensor]
    mask: np.ndarray                     # [H] uint8
    planted: List[np.ndarray] = field(default_factory=list)


def layer_inputs(wl: Workload, layer: int, device, seq_lens: Optional[Tuple[int, ...]] = None,
                 with_v: bool = True) -> LayerInputs:
    """Draw one layer's inputs for every prompt of the batch on `device`."""
    seq_lens = tuple(seq_lens) if seq_lens is not None else wl.seq_lens
    device = torch.device(device)
    mask = head_mask(wl, layer)
    G = wl.num_q_heads // wl.num_kv_heads
    H, n_kv, d, w = wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window
    gen = torch.Generator(device=device)
    out = LayerInputs([], [], [], mask, [])
    for s, L in enumerate(seq_lens):
        gen.manual_seed(layer_seed(wl, layer) * 64 + s)
        q = torch.randn((H, w, d), generator=gen, device=device, dtype=torch.float32).to(wl.dtype)
        k32 = torch.randn((n_kv, L, d), generator=gen, device=device, dtype=torch.float32)
        pos = planted_positions(wl, layer, s, L)
        pos_t = torch.from_numpy(pos).to(device)
        qf = q.float()
        for g in range(n_kv):
            chosen = [g * G + t for t in range(G) if mask[g * G + t]]
            qbar = qf[chosen].reshape(-1, d).mean(dim=0)
            delta = 3.0 * math.sqrt(d) * qbar / (qbar @ qbar)
            k32[g, pos_t] += delta
        k = k32.to(wl.dtype)
        del k32
        out.q_win.append(q)
        out.k.append(k)
        if with_v:
            out.v.append(torch.randn((n_kv, L, d), generator=gen, device=device,
                                     dtype=torch.float32).to(wl.dtype))
        out.planted.append(pos)
    return out
