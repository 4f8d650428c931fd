"""Brute-force (pure Python loops) reference for tiny sizes.

TEST INFRASTRUCTURE ONLY: used to pin the numpy oracle at tiny shapes.  Every
quantity is computed element by element with explicit loops, no BLAS and no
vectorisation, straight from the definitions the oracle follows (Sec. 2.1 and
supplementary Sec. S1.1): RMSNorm, projection with low-rank delta, rotate-half
rotation through cos/sin of p * theta^(-2i/hd), n x n causal softmax attention,
SwiGLU MLP and the two residual additions.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple


def mat(x) -> List[List[float]]:
    return [[float(v) for v in row] for row in x]


def vec(x) -> List[float]:
    return [float(v) for v in x]


def rms_norm_row(x: Sequence[float], g: Sequence[float], eps: float) -> List[float]:
    ms = sum(v * v for v in x) / len(x)
    r = 1.0 / math.sqrt(ms + eps)
    return [x[i] * r * g[i] for i in range(len(x))]


def linear_row(x: Sequence[float], w: List[List[float]], a=None, b=None, scale=1.0, bias=None) -> List[float]:
    d_out = len(w)
    y = []
    u = None
    if a is not None:
        u = [sum(x[k] * a[j][k] for k in range(len(x))) for j in range(len(a))]
    for o in range(d_out):
        acc = sum(x[k] * w[o][k] for k in range(len(x)))
        if u is not None:
            acc += scale * sum(u[j] * b[o][j] for j in range(len(u)))
        if bias is not None:
            acc += bias[o]
        y.append(acc)
    return y


def rope_vec(x: Sequence[float], p: int, theta: float) -> List[float]:
    hd = len(x)
    half = hd // 2
    out = [0.0] * hd
    for i in range(half):
        phi = p * theta ** (-(2.0 * i) / hd)
        c, s = math.cos(phi), math.sin(phi)
        out[i] = x[i] * c - x[i + half] * s
        out[i + half] = x[i + half] * c + x[i] * s
    return out


def attention(q, k, v, n_q_heads: int, n_kv_heads: int, head_dim: int):
    """q[p][j][e], k[p][g][e], v[p][g][e] nested lists -> o[p][j][e]."""
    n = len(q)
    rep = n_q_heads // n_kv_heads
    o = [[[0.0] * head_dim for _ in range(n_q_heads)] for _ in range(n)]
    for p in range(n):
        for j in range(n_q_heads):
            g = j // rep
            scores = []
            for t in range(p + 1):
                scores.append(sum(q[p][j][e] * k[t][g][e] for e in range(head_dim)) / math.sqrt(head_dim))
            m = max(scores)
            ex = [math.exp(s - m) for s in scores]
            z = sum(ex)
            for e in range(head_dim):
                o[p][j][e] = sum(ex[t] / z * v[t][g][e] for t in range(p + 1))
    return o


def decoder_layer(h, w: Dict, lora: Optional[Dict], dims, lora_scale: float = 1.0):
    """Returns (H_l, K_l, V_l) as nested lists."""
    lora = lora or {}
    n = len(h)
    nq, nkv, hd = dims.n_q_heads, dims.n_kv_heads, dims.head_dim
    W = {t: mat(w["w_" + t]) for t in ("q", "k", "v", "o", "gate", "up", "down")}
    L = {t: (mat(a), mat(b)) for t, (a, b) in lora.items()}
    bias = {t: (vec(w["bias_" + t]) if w.get("bias_" + t) is not None else None) for t in ("q", "k", "v")}

    def lin(x, t, bb=None):
        a, b = L.get(t, (None, None))
        return linear_row(x, W[t], a, b, lora_scale, bb)

    gA, gM = vec(w["attn_norm"]), vec(w["mlp_norm"])
    q, k, v = [], [], []
    for p in range(n):
        x = rms_norm_row(h[p], gA, dims.rms_eps)
        qp, kp, vp = lin(x, "q", bias["q"]), lin(x, "k", bias["k"]), lin(x, "v", bias["v"])
        q.append([rope_vec(qp[j * hd:(j + 1) * hd], p, dims.rope_theta) for j in range(nq)])
        k.append([rope_vec(kp[g * hd:(g + 1) * hd], p, dims.rope_theta) for g in range(nkv)])
        v.append([vp[g * hd:(g + 1) * hd] for g in range(nkv)])
    o = attention(q, k, v, nq, nkv, hd)
    out = []
    for p in range(n):
        flat = [o[p][j][e] for j in range(nq) for e in range(hd)]
        proj = lin(flat, "o")
        h1 = [h[p][i] + proj[i] for i in range(len(proj))]
        x2 = rms_norm_row(h1, gM, dims.rms_eps)
        gt, up = lin(x2, "gate"), lin(x2, "up")
        act = [gt[i] / (1.0 + math.exp(-gt[i])) * up[i] for i in range(len(gt))]
        dn = lin(act, "down")
        out.append([h1[i] + dn[i] for i in range(len(dn))])
    return out, k, v
