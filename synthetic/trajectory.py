"""Seeded synthetic set-up for an update trajectory (device placement only).

A whole model (every layer's weights), a base LoRA adapter, the embedding
state H_{-1}, maintained cache states (paged K/V pools and one retained
boundary state per layer) and a sequence of single-factor adapter updates.
Values are drawn on the device from a seeded torch generator (weights
N(0, 0.02), RMSNorm gains 1 + N(0, 0.02), A ~ N(0, 1/8), B ~ N(0, 0.01), each
update adds N(0, 0.005) to one B factor), so a 28-layer 7B-shaped model is
ready in seconds.  Computes no part of the method.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List

import numpy as np
import torch

from . import TARGETS, Dims, Workload, gen_block_table
from .device import canary_fill


def _randn(g: torch.Generator, shape, std: float, mean: float = 0.0) -> torch.Tensor:
    x = torch.randn(shape, generator=g, device="cuda", dtype=torch.float32)
    return (x * std + mean).to(torch.bfloat16).contiguous()


@dataclass
class TrajectorySetup:
    dims: Dims
    n_tokens: int
    weights: List[Dict[str, torch.Tensor]]
    base_lora: List[dict]
    embedding: torch.Tensor
    block_table: torch.Tensor
    n_phys: int
    updates: List[tuple]           # (layer, target) per update


def make_setup(wl: Workload, seed: int, n_tokens: int, n_updates: int) -> TrajectorySetup:
    d: Dims = wl.dims
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    weights, lora = [], []
    for l in range(d.n_layers):
        w = {"attn_norm": _randn(g, (d.d_model,), 0.02, 1.0), "mlp_norm": _randn(g, (d.d_model,), 0.02, 1.0)}
        ll = {"rank": wl.lora_rank, "scale": wl.lora_scale, "targets": {}}
        for t in TARGETS:
            d_out, d_in = d.target_shape(t)
            w["w_" + t] = _randn(g, (d_out, d_in), 0.02)
            if t in wl.lora_targets:
                ll["targets"][t] = (_randn(g, (wl.lora_rank, d_in), 1 / 8), _randn(g, (d_out, wl.lora_rank), 0.01))
        weights.append(w)
        lora.append(ll)
    emb = torch.randn((n_tokens, d.d_model), generator=g, device="cuda").to(torch.bfloat16)
    bt, n_phys = gen_block_table(wl, seed, n_tokens)
    rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(wl.config_id, 991)))
    updates = [(int(rng.integers(d.n_layers)), str(rng.choice(list(wl.lora_targets)))) for _ in range(n_updates)]
    return TrajectorySetup(d, n_tokens, weights, lora, emb, torch.from_numpy(bt).cuda(), n_phys, updates)


def update_step_norm(wl: Workload) -> float:
    """Mean l2 norm of one update's change (N(0, 0.005) on one B factor)."""
    d = wl.dims
    return float(np.mean([0.005 * np.sqrt(d.target_shape(t)[0] * wl.lora_rank) for t in wl.lora_targets]))


def make_calibration_conditions(wl: Workload, seed: int, n: int = 256) -> List[tuple]:
    """Synthetic calibration tuples (r_i, d_i, h*_i) standing in for the paper's
    calibration split, which needs trained adapters and task data.  d_i is the
    distance after k ~ U{1..8} accumulated updates (times a log-normal factor);
    the window a condition needs grows with d_i and shrinks with depth,
    h_need = floor(3 * d_i / E[d] * exp(-r_i / 8)) (0: reuse is safe), and h*_i
    is the first candidate window {0, 1, 2, 4, 8, 16, N - r_i} (each capped at
    N - r_i) at least that long."""
    N = wl.dims.n_layers
    e_d = update_step_norm(wl)
    rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(wl.config_id, 992)))
    out = []
    for _ in range(n):
        r = int(rng.integers(N))
        k = int(rng.integers(1, 9))
        dist = e_d * np.sqrt(k) * float(np.exp(rng.normal(0.0, 0.3)))
        need = int(np.floor(3.0 * dist / e_d * np.exp(-r / 8.0)))
        cands = sorted({min(h, N - r) for h in (0, 1, 2, 4, 8, 16)} | {N - r})
        h_star = next((h for h in cands if h >= need), N - r)
        out.append((r, dist, h_star))
    return out


def new_b(setup: TrajectorySetup, lora_now: List[dict], layer: int, target: str, g: torch.Generator) -> torch.Tensor:
    """The updated B factor: the current one plus N(0, 0.005)."""
    b = lora_now[layer]["targets"][target][1]
    return (b.float() + 0.005 * torch.randn(b.shape, generator=g, device="cuda")).to(torch.bfloat16).contiguous()


def make_state_buffers(setup: TrajectorySetup, page_size: int, restart_every: int = 1):
    """Paged K/V pools (canary-filled) and a boundary-state buffer at every
    retained boundary: boundaries[0] holds H_{-1}, boundaries[l] exists for l a
    multiple of restart_every and for l = N (the last layer's output)."""
    d = setup.dims
    shape = (d.n_layers, setup.n_phys, d.n_kv_heads, page_size, d.head_dim)
    k = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    v = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    canary_fill(k)
    canary_fill(v)
    bnd = [setup.embedding] + [torch.empty_like(setup.embedding) if (l % restart_every == 0 or l == d.n_layers)
                               else None for l in range(1, d.n_layers + 1)]
    return k, v, bnd
