"""Bounded stale-KV recomputation on MI355X (gfx950).

The compute lives in libcrf.so (HIP kernels behind the C ABI of
include/crf.h); this package is its thin Python binding.
"""
from ._lib import (  # noqa: F401
    CRF_BF16, CRF_F32, KERNEL_KINDS, TARGETS, Context, CrfError, KVCache, LayerWeights, LoraLayer, ModelDims,
    WindowItem, abi_version, kv_cache, last_error, layer_drift, layer_drift_noalloc, layer_weights_array, load, lora_array, make_dims,
    recompute_window, recompute_window_batched, status_string, validate_dims, validate_window, window_item,
    device_info, decode_logits,
)
