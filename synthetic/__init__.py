"""Seeded synthetic workloads for the bounded KV-window recomputation path.

This module is shared by the tests, the benchmark and the oracle checks.  It
holds the workload shapes and seeded random generators only: it computes no
part of the method (no normalisation, projection, rotation, attention or MLP
arithmetic).  Every random tensor is drawn in fp32 from its own PCG64 stream
(keyed by seed, workload id, layer and tensor id) and, for bf16 workloads,
rounded to bf16 with round-to-nearest-even so that the GPU and the oracle see
the same exactly-representable values.

The workloads stand in for the paper's Qwen2.5-1.5B / 7B experiments at 4K and
16K context (Sec. 5 setup): the paper's datasets and trained weights are not
used; only the shapes are taken from it.  The distributions are:
  boundary hidden state  N(0, 1)
  base weights           N(0, 0.02)       (second argument = std deviation)
  RMSNorm gains          1 + N(0, 0.02)
  LoRA A                 N(0, 1/8)        stored [r, d_in]
  LoRA B (old version)   N(0, 0.01)       stored [d_out, r]
  LoRA B (new version)   B_old + N(0, 0.005)
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

TARGETS: Tuple[str, ...] = ("q", "k", "v", "o", "gate", "up", "down")
ATTN_TARGETS: Tuple[str, ...] = ("q", "k", "v", "o")
# Paper's held-out trajectory seeds (Sec. S3 reproducibility); 7 is the timing seed.
PARITY_SEEDS: Tuple[int, ...] = (7, 17, 29)


@dataclass(frozen=True)
class Dims:
    """Decoder shape: N layers indexed 0..N-1 (Sec. 2.2, Eq. 1)."""
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    rms_eps: float = 1e-6
    rope_theta: float = 1e6
    dtype: str = "bf16"  # storage type of every tensor: "f32" or "bf16"

    @property
    def dq(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def dkv(self) -> int:
        return self.n_kv_heads * self.head_dim

    def target_shape(self, t: str) -> Tuple[int, int]:
        """(d_out, d_in) of projection target t (nn.Linear layout)."""
        d, dq, dkv, f = self.d_model, self.dq, self.dkv, self.d_ffn
        return {"q": (dq, d), "k": (dkv, d), "v": (dkv, d), "o": (d, dq),
                "gate": (f, d), "up": (f, d), "down": (d, f)}[t]


@dataclass(frozen=True)
class Window:
    """One recomputation request: layers [l0, l0+h) over n_tokens prefix tokens."""
    n_tokens: int
    l0: int
    h: int


@dataclass(frozen=True)
class Workload:
    name: str
    config_id: int
    dims: Dims
    windows: Tuple[Window, ...]
    lora_rank: int
    lora_targets: Tuple[str, ...]
    page_size: int = 16
    spare_pages: int = 4       # physical pages never named by the block table (canaries)
    lora_scale: float = 1.0

    @property
    def window(self) -> Window:
        assert len(self.windows) == 1
        return self.windows[0]

    def with_window(self, n_tokens=None, l0=None, h=None) -> "Workload":
        w = self.window
        nw = Window(n_tokens if n_tokens is not None else w.n_tokens,
                    l0 if l0 is not None else w.l0, h if h is not None else w.h)
        return dataclasses.replace(self, windows=(nw,))

    def with_dims(self, **kw) -> "Workload":
        return dataclasses.replace(self, dims=dataclasses.replace(self.dims, **kw))


QWEN15 = Dims(n_layers=28, d_model=1536, n_q_heads=12, n_kv_heads=2, head_dim=128, d_ffn=8960)
QWEN7 = Dims(n_layers=28, d_model=3584, n_q_heads=28, n_kv_heads=4, head_dim=128, d_ffn=18944)
TINY = Dims(n_layers=4, d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=64, d_ffn=704, dtype="f32")


def _mixed_windows(seed: int = 7) -> Tuple[Window, ...]:
    """8 ragged stale caches: n ~ U{2048..16384}, l0 ~ U{0..26}, h ~ U{1,2,3}
    clamped to the candidate clamp min(h, N - l0) of Sec. 4.1."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(5, 0, 0))))
    out = []
    for _ in range(8):
        n = int(rng.integers(2048, 16384, endpoint=True))
        l0 = int(rng.integers(0, 26, endpoint=True))
        h = int(rng.integers(1, 3, endpoint=True))
        out.append(Window(n, l0, min(h, QWEN15.n_layers - l0)))
    return tuple(out)


WORKLOADS: Dict[str, Workload] = {
    "tiny_f32": Workload("tiny_f32", 1, TINY, (Window(128, 1, 2),), 8, ATTN_TARGETS),
    "qwen15b_4k": Workload("qwen15b_4k", 2, QWEN15, (Window(4096, 10, 2),), 16, ATTN_TARGETS),
    "qwen7b_16k": Workload("qwen7b_16k", 3, QWEN7, (Window(16384, 14, 2),), 16, TARGETS),
    "qwen7b_16k_suffix": Workload("qwen7b_16k_suffix", 4, QWEN7, (Window(16384, 4, 24),), 16, TARGETS),
    "qwen15b_mixed8": Workload("qwen15b_mixed8", 5, QWEN15, _mixed_windows(), 16, ATTN_TARGETS),
}


# --------------------------------------------------------------------------- rounding

def round_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> nearest bf16 (ties to even), returned as fp32 holding the exact value."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    return round_bf16(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


# --------------------------------------------------------------------------- streams

_TENSOR_IDS = {
    "hidden": 1, "attn_norm": 2, "mlp_norm": 3, "block_table": 4, "sensitivity": 5,
    "anchors": 6, "canary": 7, "bias_q": 8, "bias_k": 9, "bias_v": 10,
    "new_tokens": 11, "final_norm": 12, "lm_head": 13,
}
for _i, _t in enumerate(TARGETS):
    _TENSOR_IDS["w_" + _t] = 20 + _i
    _TENSOR_IDS["lora_a_" + _t] = 40 + _i
    _TENSOR_IDS["lora_b_" + _t] = 60 + _i
    _TENSOR_IDS["lora_db_" + _t] = 80 + _i


def rng_for(seed: int, config_id: int, layer: int, tensor: str, sub: int = 0) -> np.random.Generator:
    """Independent PCG64 stream for (seed, workload, layer, tensor, sub)."""
    ss = np.random.SeedSequence(seed, spawn_key=(config_id, layer + 1, _TENSOR_IDS[tensor], sub))
    return np.random.Generator(np.random.PCG64(ss))


def _normal(rng: np.random.Generator, shape, std: float, mean: float = 0.0) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    if mean != 0.0:
        x += np.float32(mean)
    return x


# --------------------------------------------------------------------------- generators

def gen_hidden(wl: Workload, seed: int, n_tokens: int, item: int = 0) -> np.ndarray:
    """Boundary hidden state H_{l0-1} ~ N(0,1), [n_tokens, d_model]."""
    rng = rng_for(seed, wl.config_id, -1, "hidden", item)
    return to_storage(_normal(rng, (n_tokens, wl.dims.d_model), 1.0), wl.dims.dtype)


def gen_new_tokens(wl: Workload, seed: int, n_new: int, item: int = 0) -> np.ndarray:
    """Embedding states of tokens appended after the cached prefix, N(0,1), [n_new, d_model]."""
    rng = rng_for(seed, wl.config_id, -1, "new_tokens", item)
    return to_storage(_normal(rng, (n_new, wl.dims.d_model), 1.0), wl.dims.dtype)


def gen_head(wl: Workload, seed: int, vocab: int) -> Tuple[np.ndarray, np.ndarray]:
    """Final RMSNorm gain 1 + N(0, 0.02) [d_model] and LM head N(0, 0.02) [vocab, d_model]."""
    d = wl.dims.d_model
    g = to_storage(_normal(rng_for(seed, wl.config_id, -1, "final_norm"), (d,), 0.02, 1.0), wl.dims.dtype)
    w = to_storage(_normal(rng_for(seed, wl.config_id, -1, "lm_head"), (vocab, d), 0.02), wl.dims.dtype)
    return g, w


def gen_layer_weights(wl: Workload, seed: int, layer: int, with_bias: bool = False) -> Dict[str, np.ndarray]:
    """Frozen base weights of one decoder layer (nn.Linear layout [d_out, d_in])."""
    dm = wl.dims
    out: Dict[str, np.ndarray] = {}
    for nm in ("attn_norm", "mlp_norm"):
        out[nm] = to_storage(_normal(rng_for(seed, wl.config_id, layer, nm), (dm.d_model,), 0.02, 1.0), dm.dtype)
    for t in TARGETS:
        out["w_" + t] = to_storage(_normal(rng_for(seed, wl.config_id, layer, "w_" + t), dm.target_shape(t), 0.02),
                                   dm.dtype)
    if with_bias:
        for t in ("q", "k", "v"):
            out["bias_" + t] = to_storage(
                _normal(rng_for(seed, wl.config_id, layer, "bias_" + t), (dm.target_shape(t)[0],), 0.1), dm.dtype)
    return out


def gen_lora_layer(wl: Workload, seed: int, layer: int, version: int,
                   targets: Optional[Sequence[str]] = None, item: int = 0) -> Dict[str, Tuple[np.ndarray, np.ndarray]]:
    """LoRA factors of one layer at adapter version `version` (0 = old, k = k-th update).

    A is fixed across versions; B_k = B_{k-1} + N(0, 0.005), each step rounded to
    the storage type.  Returns {target: (A [r, d_in], B [d_out, r])}.
    """
    dm, r = wl.dims, wl.lora_rank
    targets = wl.lora_targets if targets is None else targets
    out = {}
    for t in targets:
        d_out, d_in = dm.target_shape(t)
        a = to_storage(_normal(rng_for(seed, wl.config_id, layer, "lora_a_" + t, item), (r, d_in), 0.125), dm.dtype)
        b = to_storage(_normal(rng_for(seed, wl.config_id, layer, "lora_b_" + t, item), (d_out, r), 0.01), dm.dtype)
        for k in range(1, version + 1):
            db = _normal(rng_for(seed, wl.config_id, layer, "lora_db_" + t, 1000 * item + k), (d_out, r), 0.005)
            b = to_storage(b + db, dm.dtype)
        out[t] = (a, b)
    return out


def zero_lora_like(lora: Dict[str, Tuple[np.ndarray, np.ndarray]]) -> Dict[str, Tuple[np.ndarray, np.ndarray]]:
    return {t: (a, np.zeros_like(b)) for t, (a, b) in lora.items()}


def n_logical_pages(n_tokens: int, page_size: int) -> int:
    return -(-n_tokens // page_size)


def gen_block_table(wl: Workload, seed: int, n_tokens: int, item: int = 0) -> Tuple[np.ndarray, int]:
    """Seeded permutation block table; returns (table int32[ceil(n/page)], n_physical_pages).

    The physical pool holds `spare_pages` more pages than the table names, so
    untouched pages exist to be checked.
    """
    n_log = n_logical_pages(n_tokens, wl.page_size)
    n_phys = n_log + wl.spare_pages
    perm = rng_for(seed, wl.config_id, -1, "block_table", item).permutation(n_phys).astype(np.int32)
    return np.ascontiguousarray(perm[:n_log]), n_phys


def gen_sensitivity(n_layers: int, seed: int, scale: float = 1.0) -> np.ndarray:
    """Per-layer sensitivities s_l ~ U(0, 2) * scale (stand-in for a calibration profile)."""
    rng = rng_for(seed, 5, -1, "sensitivity")
    return (rng.uniform(0.0, 2.0, size=n_layers) * scale).astype(np.float32)


def gen_anchor_versions(n_layers: int, n_versions: int, seed: int) -> np.ndarray:
    rng = rng_for(seed, 5, -1, "anchors")
    return rng.integers(0, n_versions, size=n_layers).astype(np.int32)


CANARY_BITS_BF16 = 0x7FA5  # a quiet-NaN bf16 pattern never produced by the method
CANARY_BITS_F32 = 0x7FC0A5A5
