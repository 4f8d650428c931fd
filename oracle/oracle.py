"""Oracle for bounded KV-window recomputation (CacheReforge hot path).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports this module:
only the tests, the smoke check and the benchmark's CPU-baseline leg may call
it.  It shares no code with the HIP library.

Plain, slow, obviously-correct numpy in float64.  Each function is the plain
definition of one step of ordinary decoder execution; the method claims that
recovery is exactly that execution restricted to a layer range (Sec. 4.2,
"Bounded Recovery": refreshed states come from ordinary decoder execution under
the active adapter, with no post-hoc correction).  Library matmuls are the only
primitive used; there is no fusion or reordering beyond query-blocking the
attention (which changes no result: each query row is computed independently).

Conventions (readings of points the paper leaves implicit):
  * Layers are indexed 0..N-1 and ranges are half-open (Sec. 2.2, Eq. 1;
    supplementary terminology table).
  * H_{-1} is the embedding state before layer 0; layer l maps H_{l-1} to H_l
    and writes its cache C_l = (K_l, V_l) from its input H_{l-1} alone
    (supplementary Eq. sup-layer-cache-dependency).
  * A pre-norm decoder block with RMSNorm, Q/K/V projections, rotate-half RoPE
    on Q and K, causal GQA softmax attention, output projection, residual, a
    second RMSNorm and a SwiGLU MLP with residual (supplementary Eq.
    sup-qkv-current-layer names the normalised input and the projections; the
    rotation, bias and MLP forms are the Qwen2.5 architecture the paper
    evaluates, Sec. 5 setup).
  * LoRA on target t: y = x W_t^T + scale * (x A_t^T) B_t^T, with A_t stored
    [r, d_in] and B_t stored [d_out, r]; scale defaults to 1.
  * K is cached after rotation; V unrotated.
"""
from __future__ import annotations

import math
from typing import Dict, List, Mapping, Optional, Sequence, Tuple

import numpy as np

F = np.float64
LoraLayer = Mapping[str, Tuple[np.ndarray, np.ndarray]]


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=F)


# ----------------------------------------------------------------------------- steps

def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """Normalised input (supplementary Sec. S1.1, the normalised attention input
    H-bar): y = g * x / sqrt(mean(x^2) + eps), row-wise."""
    x = _f64(x)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * _f64(g)


def lora_linear(x: np.ndarray, w: np.ndarray, lora: Optional[Tuple[np.ndarray, np.ndarray]] = None,
                scale: float = 1.0, bias: Optional[np.ndarray] = None) -> np.ndarray:
    """Frozen projection plus low-rank adapter delta (Sec. 1 / Sec. 5 setup: frozen
    base model, evolving LoRA adapter): x W^T + scale (x A^T) B^T (+ bias)."""
    x = _f64(x)
    y = x @ _f64(w).T
    if lora is not None:
        a, b = lora
        y = y + scale * ((x @ _f64(a).T) @ _f64(b).T)
    if bias is not None:
        y = y + _f64(bias)
    return y


def rope_angles(n_tokens: int, head_dim: int, theta: float) -> Tuple[np.ndarray, np.ndarray]:
    """cos/sin of phi[p, i] = p * theta^(-2i/hd), p = 0..n-1, i = 0..hd/2-1 (fp64)."""
    half = head_dim // 2
    inv_freq = theta ** (-(2.0 * np.arange(half, dtype=F)) / head_dim)
    phi = np.arange(n_tokens, dtype=F)[:, None] * inv_freq[None, :]
    return np.cos(phi), np.sin(phi)


def rope(x: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half positional rotation of x [n, heads, hd] at absolute positions
    0..n-1: pair (i, i+hd/2) is rotated by phi[p, i]."""
    x = _f64(x)
    n, _, hd = x.shape
    half = hd // 2
    c, s = rope_angles(n, hd, theta)
    c, s = c[:, None, :], s[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def rope_at(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """The same rotation at arbitrary absolute positions (x [m, heads, hd],
    positions [m]): phi[j, i] = positions[j] * theta^(-2i/hd)."""
    x = _f64(x)
    hd = x.shape[-1]
    half = hd // 2
    inv_freq = theta ** (-(2.0 * np.arange(half, dtype=F)) / hd)
    phi = _f64(positions)[:, None] * inv_freq[None, :]
    c, s = np.cos(phi)[:, None, :], np.sin(phi)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def causal_gqa_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_block: int = 1024) -> np.ndarray:
    """Standard causal softmax self-attention with grouped K/V heads (Sec. 2.1 KV
    caching; Sec. 5 setup).  q [n, nq, hd], k/v [n, nkv, hd] -> [n, nq, hd].

    Query head j reads K/V head j // (nq / nkv); scores are scaled by 1/sqrt(hd);
    query p attends to keys 0..p.  Query rows are processed in blocks only to
    bound memory; each row's softmax is computed whole.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    n, nq, hd = q.shape
    nkv = k.shape[1]
    rep = nq // nkv
    out = np.empty((n, nq, hd), dtype=F)
    scale = 1.0 / math.sqrt(hd)
    for a in range(0, n, q_block):
        b = min(n, a + q_block)
        qpos = np.arange(a, b)[:, None]
        kpos = np.arange(0, b)[None, :]
        mask = kpos > qpos
        for j in range(nq):
            g = j // rep
            s = (q[a:b, j, :] @ k[:b, g, :].T) * scale
            s[mask] = -np.inf
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[a:b, j, :] = p @ v[:b, g, :]
    return out


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


# ----------------------------------------------------------------------------- layer

def decoder_layer(h: np.ndarray, w: Mapping[str, np.ndarray], lora: Optional[LoraLayer], dims,
                  lora_scale: float = 1.0) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """One decoder layer l: returns (H_l, K_l, V_l) from H_{l-1} (supplementary Eq.
    sup-layer-cache-dependency: H_l = F_l(H_{l-1}), C_l = G_l(H_{l-1}))."""
    lora = lora or {}
    h = _f64(h)
    n = h.shape[0]
    nq, nkv, hd = dims.n_q_heads, dims.n_kv_heads, dims.head_dim

    def lin(x, t, bias=None):
        return lora_linear(x, w["w_" + t], lora.get(t), lora_scale, bias)

    x = rms_norm(h, w["attn_norm"], dims.rms_eps)
    q = lin(x, "q", w.get("bias_q")).reshape(n, nq, hd)
    k = lin(x, "k", w.get("bias_k")).reshape(n, nkv, hd)
    v = lin(x, "v", w.get("bias_v")).reshape(n, nkv, hd)
    q = rope(q, dims.rope_theta)
    k = rope(k, dims.rope_theta)
    o = causal_gqa_attention(q, k, v)
    h = h + lin(o.reshape(n, nq * hd), "o")
    x2 = rms_norm(h, w["mlp_norm"], dims.rms_eps)
    act = silu(lin(x2, "gate")) * lin(x2, "up")
    h = h + lin(act, "down")
    return h, k, v


# ----------------------------------------------------------------------------- window

def recompute_window(hidden_at_boundary: np.ndarray, weights: Mapping[int, Mapping[str, np.ndarray]],
                     lora: Mapping[int, LoraLayer], l0: int, h: int, dims, lora_scale: float = 1.0,
                     keep_hidden: bool = False):
    """Bounded recomputation R_{l0,h} (Sec. 4.2 "Executable restart"; supplementary
    Sec. S1.1 definition of R_{r,h}): feed the retained boundary state H_{l0-1}
    under the current adapter through layers l0..l0+h-1 over the complete prefix.

    Returns (H_{l0+h-1}, {l: (K_l, V_l)} for l in [l0, l0+h)[, {l: H_l}]).
    h == 0 is direct reuse: the boundary is returned unchanged and no layer is
    refreshed.
    """
    assert h >= 0 and 0 <= l0 and l0 + h <= dims.n_layers
    cur = _f64(hidden_at_boundary)
    kv: Dict[int, Tuple[np.ndarray, np.ndarray]] = {}
    hs: Dict[int, np.ndarray] = {}
    for l in range(l0, l0 + h):
        cur, k, v = decoder_layer(cur, weights[l], lora.get(l), dims, lora_scale)
        kv[l] = (k, v)
        if keep_hidden:
            hs[l] = cur
    if keep_hidden:
        return cur, kv, hs
    return cur, kv


def prefill(embeddings: np.ndarray, weights, lora, dims, lora_scale: float = 1.0):
    """Fresh full-prefill recomputation: all N layers from H_{-1} (Sec. 2.2)."""
    return recompute_window(embeddings, weights, lora, 0, dims.n_layers, dims, lora_scale, keep_hidden=True)


# ----------------------------------------------------------------------------- first decoding step

def decode_layer(h_new: np.ndarray, cache_k: np.ndarray, cache_v: np.ndarray, w: Mapping[str, np.ndarray],
                 lora: Optional[LoraLayer], dims, lora_scale: float = 1.0):
    """One decoder layer for m new tokens at positions n..n+m-1 on top of a cached
    prefix of n tokens (Sec. 2.1 KV caching): the new tokens attend to the cached
    K/V of this layer, whatever adapter version produced them, and causally to
    themselves.  Returns (H_l rows of the new tokens, their K_l, V_l)."""
    lora = lora or {}
    h = _f64(h_new)
    m = h.shape[0]
    n = cache_k.shape[0]
    nq, nkv, hd = dims.n_q_heads, dims.n_kv_heads, dims.head_dim

    def lin(x, t, bias=None):
        return lora_linear(x, w["w_" + t], lora.get(t), lora_scale, bias)

    x = rms_norm(h, w["attn_norm"], dims.rms_eps)
    pos = np.arange(n, n + m)
    q = rope_at(lin(x, "q", w.get("bias_q")).reshape(m, nq, hd), pos, dims.rope_theta)
    k = rope_at(lin(x, "k", w.get("bias_k")).reshape(m, nkv, hd), pos, dims.rope_theta)
    v = lin(x, "v", w.get("bias_v")).reshape(m, nkv, hd)
    kk = np.concatenate([_f64(cache_k), k], axis=0)
    vv = np.concatenate([_f64(cache_v), v], axis=0)
    rep = nq // nkv
    o = np.empty((m, nq, hd), dtype=F)
    for i in range(m):
        visible = n + i + 1                       # prefix plus new tokens 0..i
        for j in range(nq):
            g = j // rep
            sc = (kk[:visible, g, :] @ q[i, j, :]) / math.sqrt(hd)
            sc = np.exp(sc - sc.max())
            o[i, j, :] = (sc / sc.sum()) @ vv[:visible, g, :]
    h = h + lin(o.reshape(m, nq * hd), "o")
    x2 = rms_norm(h, w["mlp_norm"], dims.rms_eps)
    h = h + lin(silu(lin(x2, "gate")) * lin(x2, "up"), "down")
    return h, k, v


def decode_logits(x_new: np.ndarray, caches: Mapping[int, Tuple[np.ndarray, np.ndarray]], weights, lora, dims,
                  final_norm: np.ndarray, lm_head: np.ndarray, lora_scale: float = 1.0) -> np.ndarray:
    """First-step next-token logits (Sec. 3.2 "Tail Influence", z): the new
    tokens' embeddings run through all N layers over the cache (caches[l] =
    (K_l, V_l) of the prefix, possibly a mix of refreshed and historical
    layers), then the final RMSNorm and the LM head on the last new token."""
    h = _f64(x_new)
    for l in range(dims.n_layers):
        k, v = caches[l]
        h, _, _ = decode_layer(h, k, v, weights[l], lora.get(l), dims, lora_scale)
    hf = rms_norm(h[-1:], final_norm, dims.rms_eps)
    return (hf @ _f64(lm_head).T)[0]


def hybrid_caches(fresh: Mapping[int, Tuple], stale: Mapping[int, Tuple], b: int, n_layers: int):
    """Cache of boundary b: refreshed states before layer b, historical ones at b..N-1."""
    return {l: (fresh[l] if l < b else stale[l]) for l in range(n_layers)}


def tail_influence(z_by_boundary: Sequence[np.ndarray]) -> np.ndarray:
    """v_l = z^(l) - z^(l+1) and T_b = sum_{l >= b} ||v_l||_2 for b = 0..N (Eq.
    tail-influence); z_by_boundary[b] = z^(b), with z^(N) the fresh logits."""
    z = [_f64(x) for x in z_by_boundary]
    n = len(z) - 1
    norms = np.array([np.linalg.norm(z[l] - z[l + 1]) for l in range(n)])
    return np.concatenate([np.cumsum(norms[::-1])[::-1], [0.0]])


def kl_divergence(z_ref: np.ndarray, z: np.ndarray) -> float:
    """KL(softmax(z_ref) || softmax(z)) from logits, in log-sum-exp form."""
    a, b = _f64(z_ref), _f64(z)
    la = a - (a.max() + np.log(np.exp(a - a.max()).sum()))
    lb = b - (b.max() + np.log(np.exp(b - b.max()).sum()))
    return float(np.sum(np.exp(la) * (la - lb)))


# ----------------------------------------------------------------------------- drift

def layer_drift(current: Sequence[LoraLayer], versions: Sequence[Sequence[LoraLayer]],
                anchor_version: Sequence[int], sensitivity: Optional[Sequence[float]] = None,
                per_layer_only: bool = False):
    """Runtime drift and risk (Sec. 4.1 "Runtime risk", Eq. 8):
        d_l = || theta_t - theta_l^anchor ||_2,   q_l = s_l d_l.

    theta is the whole adapter (every layer's A and B of every target), so layers
    sharing an anchor version share d; per_layer_only restricts the norm to layer
    l's own slice.  Also returns the squared partials sq[v, l] of layer l's slice
    against version v.  Accumulation in float64.
    """
    n_layers = len(current)
    n_versions = len(versions)
    sq = np.zeros((n_versions, n_layers), dtype=F)
    for vi, ver in enumerate(versions):
        for l in range(n_layers):
            acc = 0.0
            for t, (a, b) in current[l].items():
                va, vb = ver[l][t]
                acc += float(np.sum((_f64(a) - _f64(va)) ** 2)) + float(np.sum((_f64(b) - _f64(vb)) ** 2))
            sq[vi, l] = acc
    d = np.empty(n_layers, dtype=F)
    for l in range(n_layers):
        av = int(anchor_version[l])
        d[l] = math.sqrt(sq[av, l] if per_layer_only else float(np.sum(sq[av, :])))
    s = np.ones(n_layers, dtype=F) if sensitivity is None else _f64(sensitivity)
    return d, s * d, sq
