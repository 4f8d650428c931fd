"""Device placement of the seeded synthetic workloads (torch tensors on the GPU).

Plumbing only: uploads the generated tensors, allocates the paged K/V pools
(filled with a canary bit pattern), and reads a layer's K/V back through the
block table.  Computes no part of the method.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import (CANARY_BITS_BF16, CANARY_BITS_F32, TARGETS, Dims, Window, Workload, gen_block_table, gen_hidden,
               gen_layer_weights, gen_lora_layer)


def tdtype(dims: Dims) -> torch.dtype:
    return torch.bfloat16 if dims.dtype == "bf16" else torch.float32


def to_dev(x: np.ndarray, dims: Dims, device="cuda") -> torch.Tensor:
    """Upload fp32 values that are exactly representable in the storage type."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device).to(tdtype(dims)).contiguous()


def canary_fill(t: torch.Tensor):
    if t.dtype == torch.bfloat16:
        t.view(torch.int16).fill_(np.int16(np.uint16(CANARY_BITS_BF16).view(np.int16)))
    else:
        t.view(torch.int32).fill_(int(np.uint32(CANARY_BITS_F32).view(np.int32)))


@dataclass
class DeviceCase:
    wl: Workload
    dims: Dims
    window: Window
    seed: int
    layers: Tuple[int, ...]
    weights: Dict[int, Dict[str, np.ndarray]] = field(default_factory=dict)     # host (fp32 holding storage values)
    lora: Dict[int, Dict[str, Tuple[np.ndarray, np.ndarray]]] = field(default_factory=dict)
    hidden: Optional[np.ndarray] = None
    block_table: Optional[np.ndarray] = None
    n_phys: int = 0
    weights_dev: List[Optional[Dict[str, torch.Tensor]]] = field(default_factory=list)
    lora_dev: List[Optional[dict]] = field(default_factory=list)
    hidden_dev: Optional[torch.Tensor] = None
    hidden_out: Optional[torch.Tensor] = None
    k_pool: Optional[torch.Tensor] = None
    v_pool: Optional[torch.Tensor] = None
    block_table_dev: Optional[torch.Tensor] = None


def lora_to_dev(lora: Dict[str, Tuple[np.ndarray, np.ndarray]], rank: int, scale: float, dims: Dims) -> dict:
    return {"rank": rank, "scale": scale,
            "targets": {t: (to_dev(a, dims), to_dev(b, dims)) for t, (a, b) in lora.items()}}


def build_case(wl: Workload, seed: int, window: Optional[Window] = None, lora_version: int = 1,
               layers: Optional[Sequence[int]] = None, with_bias: bool = False, keep_host: bool = True,
               item: int = 0, device="cuda", hidden: Optional[np.ndarray] = None,
               with_weights: bool = True) -> DeviceCase:
    """Generate and upload everything one window needs.

    layers: which layers get weights (default: the window's); the K/V pools
    always span all n_layers.  hidden: boundary state to use instead of the
    seeded N(0,1) draw (e.g. one produced by a prefill).
    """
    dims = wl.dims
    win = window or wl.windows[item]
    layers = tuple(range(win.l0, win.l0 + win.h)) if layers is None else tuple(layers)
    c = DeviceCase(wl=wl, dims=dims, window=win, seed=seed, layers=layers)
    c.weights_dev = [None] * dims.n_layers
    c.lora_dev = [None] * dims.n_layers
    for l in layers:
        lo = gen_lora_layer(wl, seed, l, lora_version, item=item)
        c.lora_dev[l] = lora_to_dev(lo, wl.lora_rank, wl.lora_scale, dims)
        if keep_host:
            c.lora[l] = lo
        if with_weights:
            w = gen_layer_weights(wl, seed, l, with_bias=with_bias)
            c.weights_dev[l] = {k: to_dev(v, dims, device) for k, v in w.items()}
            if keep_host:
                c.weights[l] = w
            del w
    h = gen_hidden(wl, seed, win.n_tokens, item) if hidden is None else hidden
    c.hidden_dev = to_dev(h, dims, device)
    c.hidden_out = torch.empty_like(c.hidden_dev)
    if keep_host:
        c.hidden = h
    bt, n_phys = gen_block_table(wl, seed, win.n_tokens, item)
    c.block_table, c.n_phys = bt, n_phys
    c.block_table_dev = torch.from_numpy(bt).to(device)
    shape = (dims.n_layers, n_phys, dims.n_kv_heads, wl.page_size, dims.head_dim)
    c.k_pool = torch.empty(shape, dtype=tdtype(dims), device=device)
    c.v_pool = torch.empty(shape, dtype=tdtype(dims), device=device)
    canary_fill(c.k_pool)
    canary_fill(c.v_pool)
    return c


def slot_index(block_table: np.ndarray, n_tokens: int, page_size: int) -> Tuple[np.ndarray, np.ndarray]:
    t = np.arange(n_tokens)
    return block_table[t // page_size].astype(np.int64), (t % page_size).astype(np.int64)


def gather_kv(pool: torch.Tensor, layer: int, block_table: np.ndarray, n_tokens: int, page_size: int,
              rows: Optional[np.ndarray] = None) -> np.ndarray:
    """[n_tokens (or len(rows)), n_kv, hd] fp64 copy of a layer's K or V, read through the block table."""
    pages, slots = slot_index(block_table, n_tokens, page_size)
    if rows is not None:
        pages, slots = pages[rows], slots[rows]
    lay = pool[layer]                                  # [n_phys, nkv, ps, hd]
    p = torch.from_numpy(pages).to(pool.device)
    s = torch.from_numpy(slots).to(pool.device)
    out = lay[p, :, s, :]                              # [n, nkv, hd]
    return out.float().cpu().numpy().astype(np.float64)


def scatter_kv(pool: torch.Tensor, layer: int, block_table: np.ndarray, page_size: int, values: np.ndarray):
    """Write [n, nkv, hd] values into a layer's pages (used to plant a stale cache)."""
    n = values.shape[0]
    pages, slots = slot_index(block_table, n, page_size)
    p = torch.from_numpy(pages).to(pool.device)
    s = torch.from_numpy(slots).to(pool.device)
    pool[layer][p, :, s, :] = torch.from_numpy(np.ascontiguousarray(values, dtype=np.float32)).to(pool.device).to(
        pool.dtype)


def canary_mask(pool: torch.Tensor) -> torch.Tensor:
    """True where the pool still holds the canary bit pattern."""
    if pool.dtype == torch.bfloat16:
        return pool.view(torch.int16) == np.int16(np.uint16(CANARY_BITS_BF16).view(np.int16))
    return pool.view(torch.int32) == int(np.uint32(CANARY_BITS_F32).view(np.int32))
