"""ctypes binding of libcrf.so (include/crf.h).

Argument marshalling only: every step of the recomputation runs inside the
library's HIP kernels.  Tensors are torch device tensors (ROCm); their device
pointers and the current HIP stream are handed to the C ABI.  There is no
fallback: if the library is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Iterable, List, Mapping, Optional, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("CRF_LIBRARY") or os.path.join(HERE, "libcrf.so")

TARGETS = ("q", "k", "v", "o", "gate", "up", "down")
NUM_TARGETS = 7

CRF_F32, CRF_BF16 = 0, 1
KERNEL_KINDS = ("norm", "lora_down", "gemm_qkv", "attn", "gemm_o", "gemm_gateup", "gemm_down", "drift", "other")

STATUS = {0: "CRF_OK", 1: "CRF_ERR_INVALID_ARG", 2: "CRF_ERR_SHAPE", 3: "CRF_ERR_RANGE", 4: "CRF_ERR_UNSUPPORTED",
          5: "CRF_ERR_WORKSPACE", 6: "CRF_ERR_HIP", 7: "CRF_ERR_DEVICE"}


class CrfError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        super().__init__(f"{STATUS.get(status, status)}: {message}")


# ----------------------------------------------------------------------------- structs

class ModelDims(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float), ("dtype", ctypes.c_int32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [("attn_norm", ctypes.c_void_p), ("mlp_norm", ctypes.c_void_p),
                ("w", ctypes.c_void_p * NUM_TARGETS),
                ("bias_q", ctypes.c_void_p), ("bias_k", ctypes.c_void_p), ("bias_v", ctypes.c_void_p)]


class LoraLayer(ctypes.Structure):
    _fields_ = [("rank", ctypes.c_int32), ("scale", ctypes.c_float),
                ("A", ctypes.c_void_p * NUM_TARGETS), ("B", ctypes.c_void_p * NUM_TARGETS)]


class KVCache(ctypes.Structure):
    _fields_ = [("k_pool", ctypes.c_void_p), ("v_pool", ctypes.c_void_p),
                ("layer_stride", ctypes.c_int64), ("page_stride", ctypes.c_int64),
                ("block_table", ctypes.c_void_p),
                ("n_pages", ctypes.c_int32), ("page_size", ctypes.c_int32), ("n_tokens", ctypes.c_int32)]


class WindowItem(ctypes.Structure):
    _fields_ = [("hidden_at_boundary", ctypes.c_void_p), ("lora", ctypes.POINTER(LoraLayer)),
                ("l0", ctypes.c_int32), ("h", ctypes.c_int32), ("kv", KVCache),
                ("hidden_out", ctypes.c_void_p)]


# ----------------------------------------------------------------------------- loading

_LIB: Optional[ctypes.CDLL] = None

EXPORTS = ("crf_status_string", "crf_abi_version", "crf_context_create", "crf_context_destroy", "crf_last_error",
           "crf_validate_dims", "crf_validate_window", "crf_recompute_window", "crf_recompute_window_batched",
           "crf_layer_drift", "crf_context_device_errors", "crf_context_set_timing", "crf_context_set_timing_classes",
           "crf_context_read_timing",
           "crf_device_info", "crf_decode_logits", "crf_layer_drift_noalloc")


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libcrf.so (once).  Raises if it is missing: there is no fallback."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise ImportError(f"libcrf.so not built at {path}; run `python -m paper_2609_30884_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_void_p
    lib.crf_status_string.restype = ctypes.c_char_p
    lib.crf_status_string.argtypes = [I32]
    lib.crf_abi_version.restype = I32
    lib.crf_last_error.restype = ctypes.c_char_p
    lib.crf_last_error.argtypes = [VP]
    lib.crf_context_create.restype = I32
    lib.crf_context_create.argtypes = [P(ModelDims), I32, I32, P(VP)]
    lib.crf_context_destroy.restype = None
    lib.crf_context_destroy.argtypes = [VP]
    lib.crf_validate_dims.restype = I32
    lib.crf_validate_dims.argtypes = [P(ModelDims)]
    lib.crf_validate_window.restype = I32
    lib.crf_validate_window.argtypes = [P(ModelDims), I32, I32, P(KVCache)]
    lib.crf_recompute_window.restype = I32
    lib.crf_recompute_window.argtypes = [VP, P(ModelDims), VP, P(LayerWeights), P(LoraLayer), I32, I32, P(KVCache),
                                         VP, VP]
    lib.crf_recompute_window_batched.restype = I32
    lib.crf_recompute_window_batched.argtypes = [VP, P(ModelDims), P(LayerWeights), I32, P(WindowItem), VP]
    lib.crf_layer_drift.restype = I32
    lib.crf_layer_drift.argtypes = [VP, P(ModelDims), P(LoraLayer), I32, P(P(LoraLayer)), P(I32), VP, I32, VP, VP,
                                    VP, VP]
    lib.crf_layer_drift_noalloc.restype = I32
    lib.crf_layer_drift_noalloc.argtypes = [P(ModelDims), P(LoraLayer), I32, P(P(LoraLayer)), P(I32), VP, I32, VP,
                                            VP, VP, VP]
    lib.crf_context_device_errors.restype = I32
    lib.crf_context_device_errors.argtypes = [VP, P(I32)]
    lib.crf_context_set_timing.restype = I32
    lib.crf_context_set_timing.argtypes = [VP, I32]
    lib.crf_context_set_timing_classes.restype = I32
    lib.crf_context_set_timing_classes.argtypes = [VP, ctypes.c_uint32]
    lib.crf_context_read_timing.restype = I32
    lib.crf_context_read_timing.argtypes = [VP, P(ctypes.c_float), P(I32), I32]
    lib.crf_decode_logits.restype = I32
    lib.crf_decode_logits.argtypes = [VP, P(ModelDims), VP, I32, P(LayerWeights), P(LoraLayer), P(KVCache), VP, VP,
                                      I32, VP, VP]
    lib.crf_device_info.restype = I32
    lib.crf_device_info.argtypes = [I32, P(I32), P(I32), ctypes.c_char_p, I32]
    _LIB = lib
    return lib


def _err(lib, ctx, st: int):
    if st != 0:
        msg = lib.crf_last_error(ctx)
        raise CrfError(st, msg.decode() if msg else "")


# ----------------------------------------------------------------------------- marshalling

def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return int(t.data_ptr())


def make_dims(n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, rms_eps=1e-6, rope_theta=1e6,
              dtype="bf16") -> ModelDims:
    return ModelDims(n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, rms_eps, rope_theta,
                     CRF_BF16 if dtype == "bf16" else CRF_F32)


def layer_weights_array(layers: Sequence[Optional[Mapping]]) -> ctypes.Array:
    """layers[l]: {"attn_norm", "mlp_norm", "w_q" ... "w_down", optional "bias_q/k/v"} of
    device tensors, or None for layers outside every window."""
    arr = (LayerWeights * len(layers))()
    for l, w in enumerate(layers):
        if w is None:
            continue
        arr[l].attn_norm = _ptr(w["attn_norm"])
        arr[l].mlp_norm = _ptr(w["mlp_norm"])
        for i, t in enumerate(TARGETS):
            arr[l].w[i] = _ptr(w["w_" + t])
        arr[l].bias_q = _ptr(w.get("bias_q"))
        arr[l].bias_k = _ptr(w.get("bias_k"))
        arr[l].bias_v = _ptr(w.get("bias_v"))
    return arr


def lora_array(layers: Optional[Sequence[Optional[Mapping]]], n_layers: int) -> Optional[ctypes.Array]:
    """layers[l]: {"rank": r, "scale": s, "targets": {name: (A [r, d_in], B [d_out, r])}} or None."""
    if layers is None:
        return None
    arr = (LoraLayer * n_layers)()
    for l, ll in enumerate(layers):
        if not ll:
            continue
        arr[l].rank = int(ll["rank"])
        arr[l].scale = float(ll.get("scale", 1.0))
        for i, t in enumerate(TARGETS):
            ab = ll["targets"].get(t)
            if ab is not None:
                arr[l].A[i] = _ptr(ab[0])
                arr[l].B[i] = _ptr(ab[1])
    return arr


def kv_cache(k_pool, v_pool, block_table, n_tokens: int, page_size: int) -> KVCache:
    """k_pool/v_pool: [n_layers, n_pages, n_kv_heads, page_size, head_dim] device tensors."""
    n_pages = int(k_pool.shape[1])
    return KVCache(_ptr(k_pool), _ptr(v_pool), int(k_pool.stride(0)), int(k_pool.stride(1)), _ptr(block_table),
                   n_pages, int(page_size), int(n_tokens))


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


# ----------------------------------------------------------------------------- API

class Context:
    """crf_context: workspace for windows of up to max_tokens tokens."""

    def __init__(self, dims: ModelDims, max_tokens: int, max_lora_rank: int = 16):
        self.lib = load()
        self.dims = dims
        h = ctypes.c_void_p()
        _err(self.lib, None, self.lib.crf_context_create(ctypes.byref(dims), int(max_tokens), int(max_lora_rank),
                                                          ctypes.byref(h)))
        self.handle = h

    def close(self):
        if getattr(self, "handle", None) and self.handle.value:
            self.lib.crf_context_destroy(self.handle)
            self.handle = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def device_errors(self) -> int:
        out = ctypes.c_int32()
        _err(self.lib, self.handle, self.lib.crf_context_device_errors(self.handle, ctypes.byref(out)))
        return int(out.value)

    def set_timing(self, on: bool, classes=None):
        """Event timing of every kernel class (on), of none, or of the named
        classes only (KERNEL_KINDS names)."""
        if classes is None:
            _err(self.lib, self.handle, self.lib.crf_context_set_timing(self.handle, 1 if on else 0))
            return
        mask = 0
        for name in classes if on else ():
            mask |= 1 << KERNEL_KINDS.index(name)
        _err(self.lib, self.handle, self.lib.crf_context_set_timing_classes(self.handle, mask))

    def read_timing(self) -> Dict[str, Tuple[float, int]]:
        n = len(KERNEL_KINDS)
        ms = (ctypes.c_float * n)()
        cnt = (ctypes.c_int32 * n)()
        _err(self.lib, self.handle, self.lib.crf_context_read_timing(self.handle, ms, cnt, n))
        return {k: (float(ms[i]), int(cnt[i])) for i, k in enumerate(KERNEL_KINDS)}


def device_info(device: int = 0) -> Dict[str, object]:
    """Compute-unit count, peak engine clock and architecture of a device."""
    lib = load()
    cu, mhz = ctypes.c_int32(), ctypes.c_int32()
    name = ctypes.create_string_buffer(64)
    _err(lib, None, lib.crf_device_info(device, ctypes.byref(cu), ctypes.byref(mhz), name, 64))
    return {"arch": name.value.decode(), "compute_units": int(cu.value), "max_sclk_mhz": int(mhz.value)}


def status_string(st: int) -> str:
    return load().crf_status_string(int(st)).decode()


def abi_version() -> int:
    return int(load().crf_abi_version())


def validate_dims(dims: ModelDims) -> int:
    return int(load().crf_validate_dims(ctypes.byref(dims)))


def validate_window(dims: ModelDims, l0: int, h: int, kv: KVCache) -> int:
    """Host-only check (no device needed); returns the status code."""
    return int(load().crf_validate_window(ctypes.byref(dims), int(l0), int(h), ctypes.byref(kv)))


def last_error(ctx: Optional[Context] = None) -> str:
    lib = load()
    return lib.crf_last_error(ctx.handle if ctx else None).decode()


def recompute_window(ctx: Context, dims: ModelDims, hidden_at_boundary, base_weights: ctypes.Array,
                     lora: Optional[ctypes.Array], l0: int, h: int, kv: KVCache, hidden_out=None, stream=None):
    """crf_recompute_window: refresh layers [l0, l0+h) of `kv` from H_{l0-1}."""
    lib = ctx.lib
    st = lib.crf_recompute_window(ctx.handle, ctypes.byref(dims), _ptr(hidden_at_boundary), base_weights,
                                  lora, int(l0), int(h), ctypes.byref(kv), _ptr(hidden_out), _stream(stream))
    _err(lib, ctx.handle, st)


def window_item(hidden_at_boundary, lora: Optional[ctypes.Array], l0: int, h: int, kv: KVCache,
                hidden_out=None) -> WindowItem:
    it = WindowItem()
    it.hidden_at_boundary = _ptr(hidden_at_boundary)
    it.lora = ctypes.cast(lora, ctypes.POINTER(LoraLayer)) if lora is not None else None
    it.l0, it.h, it.kv = int(l0), int(h), kv
    it.hidden_out = _ptr(hidden_out)
    return it


def recompute_window_batched(ctx: Context, dims: ModelDims, base_weights: ctypes.Array, items: Sequence[WindowItem],
                             stream=None):
    """crf_recompute_window_batched over independent stale caches."""
    arr = (WindowItem * len(items))(*items)
    st = ctx.lib.crf_recompute_window_batched(ctx.handle, ctypes.byref(dims), base_weights, len(items), arr,
                                              _stream(stream))
    _err(ctx.lib, ctx.handle, st)


def decode_logits(ctx: Context, dims: ModelDims, new_tokens, base_weights: ctypes.Array,
                  lora: Optional[ctypes.Array], kv: KVCache, final_norm, lm_head, logits_out, stream=None):
    """crf_decode_logits: first-step next-token logits of the last of new_tokens
    [n_new, d] over the cached prefix kv (kv.n_tokens tokens)."""
    lib = ctx.lib
    st = lib.crf_decode_logits(ctx.handle, ctypes.byref(dims), _ptr(new_tokens), int(new_tokens.shape[0]),
                               base_weights, lora, ctypes.byref(kv), _ptr(final_norm), _ptr(lm_head),
                               int(lm_head.shape[0]), _ptr(logits_out), _stream(stream))
    _err(lib, ctx.handle, st)


def layer_drift(ctx: Context, dims: ModelDims, current: ctypes.Array, versions: Sequence[ctypes.Array],
                anchor_version: Sequence[int], sensitivity, drift_out, risk_out, sq_partial_out=None,
                per_layer_only: bool = False, stream=None):
    """crf_layer_drift: d_l = ||theta_t - theta_anchor(l)||_2 and q_l = s_l d_l."""
    n_layers = dims.n_layers
    vp = (ctypes.POINTER(LoraLayer) * len(versions))(*[ctypes.cast(v, ctypes.POINTER(LoraLayer)) for v in versions])
    anc = (ctypes.c_int32 * n_layers)(*[int(a) for a in anchor_version])
    st = ctx.lib.crf_layer_drift(ctx.handle, ctypes.byref(dims), current, len(versions), vp, anc, _ptr(sensitivity),
                                 1 if per_layer_only else 0, _ptr(drift_out), _ptr(risk_out), _ptr(sq_partial_out),
                                 _stream(stream))
    _err(ctx.lib, ctx.handle, st)


def layer_drift_noalloc(dims: ModelDims, current: ctypes.Array, versions: Sequence[ctypes.Array],
                        anchor_version: Sequence[int], sensitivity, drift_out, risk_out, sq_partial_out=None,
                        per_layer_only: bool = False, stream=None):
    """crf_layer_drift_noalloc: crf_layer_drift without a context, in the library's fixed device scratch."""
    lib = load()
    n_layers = dims.n_layers
    vp = (ctypes.POINTER(LoraLayer) * len(versions))(*[ctypes.cast(v, ctypes.POINTER(LoraLayer)) for v in versions])
    anc = (ctypes.c_int32 * n_layers)(*[int(a) for a in anchor_version])
    st = lib.crf_layer_drift_noalloc(ctypes.byref(dims), current, len(versions), vp, anc, _ptr(sensitivity),
                                     1 if per_layer_only else 0, _ptr(drift_out), _ptr(risk_out),
                                     _ptr(sq_partial_out), _stream(stream))
    _err(lib, None, st)
