"""Full-size GPU parity on sampled rows against stored oracle values.

The fp64 oracle takes minutes per 7B layer at 16K tokens, so
tests/golden/make_golden.py (oracle + seeded inputs only) stores, for each
output tensor, its values at sampled token rows and the RMS of the whole
tensor.  Here the HIP path runs the full workload in the configuration the
benchmark times (the mixed batch through the batched call) and is compared on
those rows: element max-rel-to-RMS against the full-tensor RMS, and the
relative RMS error over the sampled rows.

Bounds: windows of up to three layers as everywhere (2e-2 relative RMS, 6e-2
per element).  The 24-layer suffix carries the depth-derived bound of the
bf16 error model (relative RMS error grows about as sqrt(depth); an exact
model of ideal bf16 execution reaches 2.1e-2 relative RMS and 0.11 per element
at its last layer): 3.5e-2 and 0.2.
"""
import os

import numpy as np
import pytest

import synthetic as syn
from tests.helpers import cdims

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
SEED = 7
BOUNDS = {"qwen7b_16k": (2e-2, 6e-2), "qwen15b_mixed8": (2e-2, 6e-2), "qwen7b_16k_suffix": (3.5e-2, 0.2)}


def _golden(name, item):
    path = os.path.join(GOLDEN, f"{name}_seed{SEED}_item{item}.npz")
    if not os.path.exists(path):
        pytest.skip(f"stored oracle samples {os.path.basename(path)} not generated")
    return np.load(path)


def _compare(case, gold, label, bounds):
    from synthetic.device import gather_kv
    rows = gold["rows"]
    n, ps = case.window.n_tokens, case.wl.page_size
    errs = {}
    for key in gold.files:
        if not key.endswith("_rows") or key == "rows":
            continue
        nm = key[:-5]
        ref = gold[key].astype(np.float64)
        rms = float(gold[nm + "_rms"])
        if nm == "hidden_out":
            got = case.hidden_out[torch.from_numpy(rows).cuda()].float().cpu().numpy().astype(np.float64)
        else:
            layer = int(nm[1:])
            pool = case.k_pool if nm[0] == "K" else case.v_pool
            got = gather_kv(pool, layer, case.block_table, n, ps, rows)
        e = got - ref
        errs[nm] = (float(np.sqrt(np.mean(e * e))) / rms, float(np.max(np.abs(e))) / rms)
    print(f"[parity] {label} (rms-rel, elem) " + " ".join(f"{k}=({a:.2e},{b:.2e})" for k, (a, b) in errs.items()),
          flush=True)
    bad = {k: v for k, v in errs.items() if not (v[0] <= bounds[0] and v[1] <= bounds[1])}
    assert not bad, f"{label}: above {bounds}: {bad}"


@pytest.mark.parametrize("name", ["qwen7b_16k", "qwen7b_16k_suffix"])
def test_full_size_window(name):
    from synthetic.device import build_case
    from tests.helpers import run_gpu_window
    gold = _golden(name, 0)
    wl = syn.WORKLOADS[name]
    print(f"[case] {name} full size n={wl.window.n_tokens} window=[{wl.window.l0},{wl.window.l0 + wl.window.h})",
          flush=True)
    case = build_case(wl, SEED, keep_host=False)
    ctx = run_gpu_window(case)
    torch.cuda.synchronize()
    assert ctx.device_errors() == 0
    _compare(case, gold, name, BOUNDS[name])


def test_full_size_mixed_batch():
    import paper_2609_30884_amd as crf
    from synthetic.device import build_case
    wl = syn.WORKLOADS["qwen15b_mixed8"]
    golds = [_golden(wl.name, i) for i in range(len(wl.windows))]
    layers = sorted({l for w in wl.windows for l in range(w.l0, w.l0 + w.h)})
    cases = [build_case(wl, SEED, window=w, item=i, layers=layers, keep_host=False, with_weights=(i == 0))
             for i, w in enumerate(wl.windows)]
    cd = cdims(wl.dims)
    ctx = crf.Context(cd, max(w.n_tokens for w in wl.windows), wl.lora_rank)
    keep, items = [], []
    for c in cases:
        la = crf.lora_array(c.lora_dev, wl.dims.n_layers)
        keep.append(la)
        kv = crf.kv_cache(c.k_pool, c.v_pool, c.block_table_dev, c.window.n_tokens, wl.page_size)
        items.append(crf.window_item(c.hidden_dev, la, c.window.l0, c.window.h, kv, c.hidden_out))
    crf.recompute_window_batched(ctx, cd, crf.layer_weights_array(cases[0].weights_dev), items)
    torch.cuda.synchronize()
    assert ctx.device_errors() == 0
    for i, (c, g) in enumerate(zip(cases, golds)):
        _compare(c, g, f"mixed item {i} n={c.window.n_tokens} [{c.window.l0},{c.window.l0 + c.window.h})",
                 BOUNDS[wl.name])
