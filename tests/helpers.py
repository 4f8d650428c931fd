"""Shared test plumbing: run the HIP path through the C ABI on a synthetic case
and run the oracle on the same host values."""
from __future__ import annotations

import numpy as np

import synthetic as syn

# Per output tensor T (each refreshed layer's K and V, and the window output):
#   rms-relative error      ||T_gpu - T_ref||_2 / ||T_ref||_2
#   element max-rel-to-RMS  max_i |T_gpu,i - T_ref,i| / rms(T_ref)
# fp32: both <= 1e-4.  bf16: rms-relative <= 2e-2; the element metric is bounded
# by what ideal bf16 execution reaches on these workloads (an exact CPU model of
# bf16 storage with fp32 accumulation gives up to 3.2e-2 on a two-layer 7B
# window), with headroom: 6e-2 for windows of up to three layers.
TOL = {"f32": 1e-4, "bf16": 2e-2}
TOL_ELEM = {"f32": 1e-4, "bf16": 6e-2}


def rel_to_rms(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    rms = np.sqrt(np.mean(ref * ref))
    return float(np.max(np.abs(got - ref)) / rms)


def rms_rel(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.sqrt(np.mean((got - ref) ** 2) / np.mean(ref * ref)))


def bits_equal(a, b) -> bool:
    """Bitwise tensor equality (canary patterns are NaNs, so == does not work)."""
    import torch
    it = {torch.bfloat16: torch.int16, torch.float16: torch.int16, torch.float32: torch.int32}[a.dtype]
    return bool(torch.equal(a.view(it), b.view(it)))


def cdims(dims: syn.Dims):
    import paper_2609_30884_amd as crf
    return crf.make_dims(dims.n_layers, dims.d_model, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.d_ffn,
                         dims.rms_eps, dims.rope_theta, dims.dtype)


def run_gpu_window(case, ctx=None, l0=None, h=None, lora_dev=None, hidden_out=True, stream=None):
    """crf_recompute_window on a synthetic.device.DeviceCase; returns the context."""
    import paper_2609_30884_amd as crf
    dims = case.dims
    cd = cdims(dims)
    win = case.window
    l0 = win.l0 if l0 is None else l0
    h = win.h if h is None else h
    if ctx is None:
        ctx = crf.Context(cd, max(win.n_tokens, 1), case.wl.lora_rank)
    kv = crf.kv_cache(case.k_pool, case.v_pool, case.block_table_dev, win.n_tokens, case.wl.page_size)
    lora = crf.lora_array(case.lora_dev if lora_dev is None else lora_dev, dims.n_layers)
    crf.recompute_window(ctx, cd, case.hidden_dev, crf.layer_weights_array(case.weights_dev), lora, l0, h, kv,
                         case.hidden_out if hidden_out else None, stream)
    return ctx


def oracle_window(case, l0=None, h=None, lora=None):
    from oracle import oracle as O
    win = case.window
    l0 = win.l0 if l0 is None else l0
    h = win.h if h is None else h
    return O.recompute_window(case.hidden, case.weights, case.lora if lora is None else lora, l0, h, case.dims,
                              case.wl.lora_scale)


def gpu_kv(case, layer, rows=None):
    from synthetic.device import gather_kv
    n = case.window.n_tokens
    return (gather_kv(case.k_pool, layer, case.block_table, n, case.wl.page_size, rows),
            gather_kv(case.v_pool, layer, case.block_table, n, case.wl.page_size, rows))


def assert_window_parity(case, out_ref, kv_ref, tol=None, tol_elem=None, label=""):
    """Element-by-element parity of every refreshed K/V layer and hidden_out."""
    dt = case.dims.dtype
    tol = TOL[dt] if tol is None else tol
    tol_elem = TOL_ELEM[dt] if tol_elem is None else tol_elem
    pairs = {}
    for l, (k_ref, v_ref) in kv_ref.items():
        k, v = gpu_kv(case, l)
        pairs[f"K{l}"] = (k, k_ref)
        pairs[f"V{l}"] = (v, v_ref)
    pairs["hidden_out"] = (case.hidden_out.float().cpu().numpy(), out_ref)
    errs = {k: (rms_rel(g, r), rel_to_rms(g, r)) for k, (g, r) in pairs.items()}
    print(f"[parity] {label} (rms-rel, elem) " + " ".join(f"{k}=({a:.2e},{b:.2e})" for k, (a, b) in errs.items()),
          flush=True)
    bad = {k: v for k, v in errs.items() if not (v[0] <= tol and v[1] <= tol_elem)}
    assert not bad, f"{label}: errors above ({tol}, {tol_elem}): {bad}"
    return {k: v[0] for k, v in errs.items()}
