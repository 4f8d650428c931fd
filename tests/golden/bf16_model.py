"""Error model of ideal bf16 execution of a recomputation window.

This script justifies the bf16 parity bounds; it is not a reference for the
GPU path (that is the fp64 oracle).  It runs the same window as the oracle,
but in fp32 arithmetic with every tensor that the HIP path keeps in bf16
rounded to bf16 (round to nearest even) at the point where it is stored:

  normalised inputs X, X2; LoRA down-projections U; stored queries Q (scaled
  by log2(e)/sqrt(hd) before rounding); refreshed K and V; the attention
  probabilities that enter the P.V product (the row sums use the fp32 ones);
  the attention output; the SwiGLU output; the window output.

The residual stream stays fp32 inside the window, as on the GPU.  Comparing
this model with the fp64 oracle gives the error that bf16 storage alone
causes, i.e. what a faithful bf16 pipeline reaches; the parity tests bound the
GPU's error in terms of it.  With rounding switched off the model equals the
oracle to fp32 accuracy (tests/test_bf16_model.py checks this).

    OPENBLAS_NUM_THREADS=8 python tests/golden/bf16_model.py qwen15b_4k qwen7b_16k qwen7b_16k_suffix

writes tests/golden/bf16_model_errors.json: per workload and output tensor
(each refreshed layer's K and V, and the window output) the relative RMS
error ||T - T_ref||/||T_ref|| and the element metric max|T - T_ref|/rms(T_ref)
of the model against the oracle, on the seed-7 inputs.
"""
from __future__ import annotations

import json
import math
import os
import sys
import time
from typing import Callable, Dict, Mapping, Optional, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import synthetic as syn  # noqa: E402
from oracle import oracle as O  # noqa: E402

F32 = np.float32
SEED = 7
OUT = os.path.join(HERE, "bf16_model_errors.json")


def _ident(x):
    return np.asarray(x, F32)


def _bf16(x):
    return syn.round_bf16(np.asarray(x, F32))


# Deviations from ideal execution that the tests plant to see which of them
# the parity check on the model's RMS error notices: an extra bf16 rounding of
# the residual stream after each residual update, or one of the model's
# rounding points left out (the tensor kept in fp32).
ROUNDING_POINTS = ("x", "u", "q", "k", "v", "p", "attn", "act")
VARIANTS = ("resid_bf16",) + tuple("skip_" + r for r in ROUNDING_POINTS)


def model_layer(h: np.ndarray, w: Mapping[str, np.ndarray], lora, dims, scale: float = 1.0,
                rnd: Callable = _bf16, first: bool = True, variant: str = ""):
    """One decoder layer as the kernels execute it: returns (H_l fp32, K_l, V_l).
    variant: one of VARIANTS, or "" for ideal execution."""
    assert variant in ("",) + VARIANTS, variant
    rres = rnd if variant == "resid_bf16" else _ident
    r_ = {pt: (_ident if variant == "skip_" + pt else rnd) for pt in ROUNDING_POINTS}
    lora = lora or {}
    h = np.asarray(h, F32)
    n = h.shape[0]
    nq, nkv, hd = dims.n_q_heads, dims.n_kv_heads, dims.head_dim
    half = hd // 2

    def norm(x, g):
        ms = np.mean(x * x, axis=1, keepdims=True, dtype=F32)
        return r_["x"](x * (F32(1.0) / np.sqrt(ms + F32(dims.rms_eps))) * np.asarray(g, F32))

    def lin(x, t, bias=None):
        y = x @ np.asarray(w["w_" + t], F32).T
        if t in lora:
            a, b = lora[t]
            u = r_["u"](F32(scale) * (x @ np.asarray(a, F32).T))
            y = y + u @ np.asarray(b, F32).T
        if bias is not None:
            y = y + np.asarray(bias, F32)
        return y

    inv_freq = dims.rope_theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / hd)
    ang = np.arange(n, dtype=np.float64)[:, None] * inv_freq[None, :]
    cs, sn = np.cos(ang).astype(F32)[:, None, :], np.sin(ang).astype(F32)[:, None, :]

    def rope(x):
        x1, x2 = x[..., :half], x[..., half:]
        return np.concatenate([x1 * cs - x2 * sn, x2 * cs + x1 * sn], axis=-1)

    x = norm(h, w["attn_norm"])
    c2 = F32(1.4426950408889634 / math.sqrt(hd))
    q = r_["q"](rope(lin(x, "q", w.get("bias_q")).reshape(n, nq, hd)) * c2)
    k = r_["k"](rope(lin(x, "k", w.get("bias_k")).reshape(n, nkv, hd)))
    v = r_["v"](lin(x, "v", w.get("bias_v")).reshape(n, nkv, hd))
    o = np.empty((n, nq, hd), F32)
    rep = nq // nkv
    blk = 512
    for a0 in range(0, n, blk):
        b0 = min(n, a0 + blk)
        mask = np.arange(b0)[None, :] > np.arange(a0, b0)[:, None]
        for j in range(nq):
            g = j // rep
            s = q[a0:b0, j, :] @ k[:b0, g, :].T          # log2 units
            s[mask] = -np.inf
            p = np.exp2(s - s.max(axis=1, keepdims=True))
            l_ = p.sum(axis=1, keepdims=True, dtype=F32)
            o[a0:b0, j, :] = (r_["p"](p) @ v[:b0, g, :]) / l_
    attn = r_["attn"](o.reshape(n, nq * hd))
    h = rres(h + lin(attn, "o"))
    x2 = norm(h, w["mlp_norm"])
    gt, up = lin(x2, "gate"), lin(x2, "up")
    act = r_["act"](gt / (F32(1.0) + np.exp(-gt)) * up)
    h = rres(h + lin(act, "down"))
    return h, k, v


def errors(got: np.ndarray, ref: np.ndarray) -> Tuple[float, float]:
    """(relative RMS error, element max-rel-to-RMS) of got against ref."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    rms = math.sqrt(float(np.mean(ref * ref)))
    e = got - ref
    return math.sqrt(float(np.mean(e * e))) / rms, float(np.max(np.abs(e))) / rms


def window_errors(wl: syn.Workload, item: int = 0, seed: int = SEED, rnd: Callable = _bf16,
                  n_tokens: Optional[int] = None, log=None, variant: str = "") -> Dict[str, Tuple[float, float]]:
    """Model vs oracle errors for one window of a workload (optionally on the
    first n_tokens of its prefix, optionally with a planted deviation)."""
    win = wl.windows[item]
    n = win.n_tokens if n_tokens is None else n_tokens
    dims = wl.dims
    hb = syn.gen_hidden(wl, seed, win.n_tokens, item)[:n]
    ref = hb.astype(np.float64)
    cur = hb.astype(F32)
    out: Dict[str, Tuple[float, float]] = {}
    for l in range(win.l0, win.l0 + win.h):
        w = syn.gen_layer_weights(wl, seed, l)
        lo = syn.gen_lora_layer(wl, seed, l, 1, item=item)
        t0 = time.perf_counter()
        ref, kr, vr = O.decoder_layer(ref, w, lo, dims, wl.lora_scale)
        t1 = time.perf_counter()
        cur, km, vm = model_layer(cur, w, lo, dims, wl.lora_scale, rnd, variant=variant)
        out[f"K{l}"] = errors(km, kr)
        out[f"V{l}"] = errors(vm, vr)
        if log:
            log(f"  {wl.name} item {item} layer {l}: oracle {t1 - t0:.1f}s model {time.perf_counter() - t1:.1f}s "
                f"K {out[f'K{l}'][1]:.3e} V {out[f'V{l}'][1]:.3e}")
        del w, lo, kr, vr, km, vm
    out["hidden_out"] = errors(rnd(cur), ref)
    return out


def main(names):
    res = json.load(open(OUT)) if os.path.exists(OUT) else {}
    for name in names:
        wl = syn.WORKLOADS[name]
        t0 = time.perf_counter()
        e = window_errors(wl, 0, log=lambda s: print(s, flush=True))
        res[name] = {"seed": SEED, "n_tokens": wl.windows[0].n_tokens, "l0": wl.windows[0].l0,
                     "h": wl.windows[0].h,
                     "errors": {k: {"rms_rel": a, "elem": b} for k, (a, b) in e.items()}}
        json.dump(res, open(OUT, "w"), indent=1, sort_keys=True)
        print(f"{name}: {time.perf_counter() - t0:.0f}s, wrote {OUT}", flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or ["qwen15b_4k"])
