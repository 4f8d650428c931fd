"""Write sampled oracle outputs for the full-size workloads.

Calls only the oracle and the seeded input generators.  For each workload the
whole window is computed by the fp64 oracle; what is stored is, per output
tensor (every refreshed layer's K and V, and the window output), the values at
a fixed set of sampled token rows and the RMS of the whole tensor, so a GPU
test can compute the element metric and the relative RMS error on the samples
against the full-tensor RMS.

    OPENBLAS_NUM_THREADS=6 python tests/golden/make_golden.py qwen7b_16k_suffix

(The 7B-shaped 16K window and the 8-item mixed batch are compared on whole
tensors against the oracle run next to the GPU, so they need no stored
samples.)
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import synthetic as syn  # noqa: E402
from oracle import oracle as O  # noqa: E402

SEED = 7
N_SAMPLES = 16
# layers whose K/V are stored for the 24-layer suffix: all of them
SUFFIX_KV_LAYERS = tuple(range(4, 28))


def sample_rows(n: int) -> np.ndarray:
    """First and last rows, tile and page edges, and seeded interior rows."""
    fixed = {0, 1, 15, 16, 63, 64, 127, 128, n - 1, n - 2}
    rng = np.random.default_rng(12345 + n)
    extra = rng.choice(n, size=N_SAMPLES, replace=False)
    return np.array(sorted({r for r in fixed if 0 <= r < n} | set(int(x) for x in extra)), dtype=np.int64)


def window_outputs(wl: syn.Workload, item: int, kv_layers=None):
    win = wl.windows[item]
    dims = wl.dims
    h = syn.gen_hidden(wl, SEED, win.n_tokens, item)
    cur = h.astype(np.float64)
    out = {}
    rows = sample_rows(win.n_tokens)
    for l in range(win.l0, win.l0 + win.h):
        w = syn.gen_layer_weights(wl, SEED, l)
        lo = syn.gen_lora_layer(wl, SEED, l, 1, item=item)
        t0 = time.perf_counter()
        cur, k, v = O.decoder_layer(cur, w, lo, dims, wl.lora_scale)
        print(f"  {wl.name} item {item} layer {l}: {time.perf_counter() - t0:.1f}s", flush=True)
        if kv_layers is None or l in kv_layers:
            for nm, t in (("K", k), ("V", v)):
                out[f"{nm}{l}_rows"] = t[rows].astype(np.float32)
                out[f"{nm}{l}_rms"] = np.array(np.sqrt(np.mean(t * t)))
        del w, lo, k, v
    out["hidden_out_rows"] = cur[rows].astype(np.float32)
    out["hidden_out_rms"] = np.array(np.sqrt(np.mean(cur * cur)))
    out["rows"] = rows
    return out


def main(names):
    for name in names:
        wl = syn.WORKLOADS[name]
        t0 = time.perf_counter()
        for item in range(len(wl.windows)):
            kv_layers = SUFFIX_KV_LAYERS if name == "qwen7b_16k_suffix" else None
            out = window_outputs(wl, item, kv_layers)
            path = os.path.join(HERE, f"{name}_seed{SEED}_item{item}.npz")
            np.savez_compressed(path, **out)
            print(f"wrote {path}", flush=True)
        print(f"{name}: {time.perf_counter() - t0:.0f}s", flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or ["qwen7b_16k_suffix"])
