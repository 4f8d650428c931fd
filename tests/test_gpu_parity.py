"""GPU parity of the HIP path (through the C ABI) against the oracle.

Tolerances per output tensor (see tests/helpers.py): fp32 1e-4 per element;
bf16 2e-2 relative RMS error and 6e-2 per element.  Every K/V layer of the window and
the window's output hidden state are compared element by element; layers
outside the window and pages outside the block table must keep their canary
bits.
"""
import numpy as np
import pytest

import synthetic as syn
from tests.helpers import (TOL, assert_window_parity, bits_equal, cdims, gpu_kv, oracle_window, rel_to_rms,
                           run_gpu_window)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    import paper_2609_30884_amd as crf
    crf.load()  # fails loudly if the HIP library is missing
    yield


def _untouched(case, layers_refreshed):
    """Pages outside the table: canary in every layer; table pages of layers
    outside the window: canary."""
    from synthetic.device import canary_mask
    spare = np.setdiff1d(np.arange(case.n_phys), case.block_table)
    for pool in (case.k_pool, case.v_pool):
        cm = canary_mask(pool)
        if len(spare):
            assert bool(cm[:, torch.from_numpy(spare).to(pool.device)].all()), "spare page written"
        for l in range(case.dims.n_layers):
            if l not in layers_refreshed:
                assert bool(cm[l].all()), f"layer {l} outside the window written"
        # slots past n_tokens in the last page stay untouched
        n, ps = case.window.n_tokens, case.wl.page_size
        if n % ps:
            last = int(case.block_table[-1])
            for l in layers_refreshed:
                assert bool(cm[l, last, :, n % ps:, :].all()), "slot past n_tokens written"


# ----------------------------------------------------------------------------- fp32 tiny workload

def test_tiny_f32_stale_cache_refresh():
    """Prefill under the old adapter plants a stale cache; the GPU refreshes
    layers [1, 3) under the new one (Sec. 4.2)."""
    from oracle import oracle as O
    from synthetic.device import build_case, scatter_kv
    wl = syn.WORKLOADS["tiny_f32"]
    seed = 7
    dims = wl.dims
    emb = syn.gen_hidden(wl, seed, wl.window.n_tokens)
    W = {l: syn.gen_layer_weights(wl, seed, l) for l in range(dims.n_layers)}
    L_old = {l: syn.gen_lora_layer(wl, seed, l, 0) for l in range(dims.n_layers)}
    _, KV_old, H_old = O.prefill(emb, W, L_old, dims)
    case = build_case(wl, seed, hidden=syn.to_storage(H_old[0].astype(np.float32), "f32"))
    for l in range(dims.n_layers):
        scatter_kv(case.k_pool, l, case.block_table, wl.page_size, KV_old[l][0])
        scatter_kv(case.v_pool, l, case.block_table, wl.page_size, KV_old[l][1])
    before = {l: (case.k_pool[l].clone(), case.v_pool[l].clone()) for l in (0, 3)}
    print("[case] tiny_f32 stale refresh [1,3)", flush=True)
    run_gpu_window(case)
    torch.cuda.synchronize()
    out, kv = oracle_window(case)
    errs = assert_window_parity(case, out, kv, label="tiny_f32")
    for l in (0, 3):
        assert bits_equal(case.k_pool[l], before[l][0]) and bits_equal(case.v_pool[l], before[l][1])
    # the refreshed layers really changed relative to the stale cache
    k1, _ = gpu_kv(case, 1)
    assert rel_to_rms(k1, KV_old[1][0]) > 10 * TOL["f32"]


def test_tiny_f32_exact_suffix_equals_fresh_prefill():
    """Recomputing the whole affected suffix [l0, N) from the retained boundary
    reproduces fresh prefill under the new adapter when the update sits at
    layers >= l0 (Sec. 2.2, exact affected-suffix recomputation)."""
    from oracle import oracle as O
    from synthetic.device import build_case, lora_to_dev
    wl = syn.WORKLOADS["tiny_f32"]
    seed, l0 = 17, 2
    dims = wl.dims
    emb = syn.gen_hidden(wl, seed, wl.window.n_tokens)
    W = {l: syn.gen_layer_weights(wl, seed, l) for l in range(dims.n_layers)}
    L_old = {l: syn.gen_lora_layer(wl, seed, l, 0) for l in range(dims.n_layers)}
    L_new = {l: (syn.gen_lora_layer(wl, seed, l, 1) if l >= l0 else L_old[l]) for l in range(dims.n_layers)}
    _, _, H_old = O.prefill(emb, W, L_old, dims)
    Hn_new, KV_new, _ = O.prefill(emb, W, L_new, dims)
    case = build_case(wl, seed, window=syn.Window(wl.window.n_tokens, l0, dims.n_layers - l0),
                      hidden=syn.to_storage(H_old[l0 - 1].astype(np.float32), "f32"))
    run_gpu_window(case)
    torch.cuda.synchronize()
    assert_window_parity(case, Hn_new, {l: KV_new[l] for l in range(l0, dims.n_layers)}, label="tiny exact suffix")


# ----------------------------------------------------------------------------- bf16 workloads

@pytest.mark.parametrize("name,n,seed", [
    ("qwen15b_4k", 1000, 7),      # ragged: not a multiple of the tile sizes or the page size
    ("qwen15b_4k", 4096, 17),     # the full 1.5B-shaped 4K window
    ("qwen7b_16k", 333, 29),      # 7B shapes, short ragged prefix
])
def test_bf16_window_parity(name, n, seed):
    from synthetic.device import build_case
    wl = syn.WORKLOADS[name].with_window(n_tokens=n)
    case = build_case(wl, seed)
    print(f"[case] {name} n={n} seed={seed} window=[{wl.window.l0},{wl.window.l0 + wl.window.h})", flush=True)
    run_gpu_window(case)
    torch.cuda.synchronize()
    out, kv = oracle_window(case)
    assert_window_parity(case, out, kv, label=f"{name} n={n}")
    _untouched(case, set(kv))


@pytest.mark.parametrize("page_size,hd,nq,nkv,n", [
    (8, 128, 12, 2, 700),    # runtime page size; two KV heads (four XCDs per KV head)
    (1, 64, 12, 6, 300),     # one-token pages, head_dim 64, six KV heads (plain launch order)
    (32, 64, 8, 2, 1100),    # 32-token pages, head_dim 64
    # one-token pages past the 2048 page bases a workgroup stages at a time:
    # the later query blocks refill their page bases mid-way
    (1, 128, 8, 2, 2500),
    (1, 64, 12, 6, 4200),
])
def test_bf16_page_sizes_and_head_shapes(page_size, hd, nq, nkv, n):
    """Paged attention and the K/V-writing epilogue with page sizes other than
    16, head_dim 64 and KV-head counts that do and do not divide the XCD count."""
    import dataclasses
    from synthetic.device import build_case
    wl = dataclasses.replace(syn.WORKLOADS["qwen15b_4k"], page_size=page_size).with_dims(
        n_layers=4, d_model=768, n_q_heads=nq, n_kv_heads=nkv, head_dim=hd, d_ffn=2048).with_window(
        n_tokens=n, l0=1, h=2)
    print(f"[case] page_size={page_size} hd={hd} nq={nq} nkv={nkv} n={n}", flush=True)
    case = build_case(wl, 11)
    run_gpu_window(case)
    torch.cuda.synchronize()
    out, kv = oracle_window(case)
    assert_window_parity(case, out, kv, label=f"ps={page_size} hd={hd} {nq}/{nkv} n={n}")
    _untouched(case, set(kv))


@pytest.mark.parametrize("name,n,l0,h,seed", [
    ("qwen15b_4k", 1000, 10, 2, 7),
    ("qwen15b_4k", 600, 5, 1, 17),     # a one-layer window is all tail
    ("qwen7b_16k", 333, 14, 2, 29),
])
def test_bf16_kv_only_tail_layer(name, n, l0, h, seed):
    """Without hidden_out the last window layer runs only its K/V projections
    (its cache entry depends on its input alone, supplementary Eq.
    sup-layer-cache-dependency): every page written is bitwise the full run's,
    and within tolerance of the oracle."""
    from synthetic.device import build_case, canary_fill
    wl = syn.WORKLOADS[name].with_window(n_tokens=n, l0=l0, h=h)
    case = build_case(wl, seed)
    print(f"[case] kv-only tail {name} n={n} window=[{l0},{l0 + h}) seed={seed}", flush=True)
    ctx = run_gpu_window(case)
    torch.cuda.synchronize()
    k_full, v_full, h_full = case.k_pool.clone(), case.v_pool.clone(), case.hidden_out.clone()
    canary_fill(case.k_pool)
    canary_fill(case.v_pool)
    run_gpu_window(case, ctx=ctx, hidden_out=False)
    torch.cuda.synchronize()
    assert bits_equal(case.k_pool, k_full) and bits_equal(case.v_pool, v_full)
    assert bits_equal(case.hidden_out, h_full)      # not written by the second call
    out, kv = oracle_window(case)
    assert_window_parity(case, out, kv, label=f"kv-only tail {name} n={n}")
    _untouched(case, set(kv))


def test_bf16_qkv_bias_and_rank8():
    """Optional q/k/v biases and a rank-8 adapter on the bf16 path."""
    from synthetic.device import build_case
    import dataclasses
    wl = dataclasses.replace(syn.WORKLOADS["qwen15b_4k"].with_window(n_tokens=300, l0=3, h=1), lora_rank=8,
                             lora_scale=0.5, lora_targets=syn.TARGETS)
    case = build_case(wl, 7, with_bias=True)
    run_gpu_window(case)
    torch.cuda.synchronize()
    out, kv = oracle_window(case)
    assert_window_parity(case, out, kv, label="bias+rank8")


def test_bf16_deterministic_and_h0_noop():
    from synthetic.device import build_case
    wl = syn.WORKLOADS["qwen15b_4k"].with_window(n_tokens=777)
    case = build_case(wl, 29)
    ctx = run_gpu_window(case)
    k1, v1 = (t.clone() for t in (case.k_pool, case.v_pool))
    h1 = case.hidden_out.clone()
    run_gpu_window(case, ctx=ctx)
    torch.cuda.synchronize()
    assert bits_equal(case.k_pool, k1) and bits_equal(case.v_pool, v1) and bits_equal(case.hidden_out, h1)
    # h = 0 is direct reuse: nothing is written
    case.hidden_out.zero_()
    run_gpu_window(case, ctx=ctx, h=0)
    torch.cuda.synchronize()
    assert bits_equal(case.k_pool, k1) and bool((case.hidden_out == 0).all())


def test_bf16_query_only_update_keeps_same_layer_kv():
    """A query/output/MLP update at layer s leaves the K/V written at s
    unchanged (supplementary Eq. sup-first-invalid-cache-layer)."""
    from synthetic.device import build_case
    wl = syn.WORKLOADS["qwen15b_4k"].with_window(n_tokens=500, l0=5, h=1)
    case = build_case(wl, 7, lora_version=0)
    ctx = run_gpu_window(case)
    k0, v0 = gpu_kv(case, 5)
    h0 = case.hidden_out.clone()
    # move only B_q and B_o to the next version
    new = syn.gen_lora_layer(wl, 7, 5, 3)
    lo = dict(case.lora_dev[5])
    tg = dict(lo["targets"])
    from synthetic.device import to_dev
    for t in ("q", "o"):
        tg[t] = (tg[t][0], to_dev(new[t][1], wl.dims))
    lo["targets"] = tg
    lora_dev = list(case.lora_dev)
    lora_dev[5] = lo
    run_gpu_window(case, ctx=ctx, lora_dev=lora_dev)
    torch.cuda.synchronize()
    k1, v1 = gpu_kv(case, 5)
    assert np.array_equal(k0, k1) and np.array_equal(v0, v1)
    assert not torch.equal(case.hidden_out, h0)


def test_block_table_entry_out_of_range_is_caught():
    """A bad block table entry is skipped by the kernels' own bounds checks and
    reported through the device error flag; other pages are still written."""
    from synthetic.device import build_case
    wl = syn.WORKLOADS["qwen15b_4k"].with_window(n_tokens=256, l0=0, h=1)
    case = build_case(wl, 7)
    bad = case.block_table.copy()
    bad[3] = case.n_phys + 5
    case.block_table_dev = torch.from_numpy(bad).to("cuda")
    ctx = run_gpu_window(case)
    flags = ctx.device_errors()
    assert flags & 1
    assert ctx.device_errors() == 0  # cleared by the read
    from synthetic.device import canary_mask
    cm = canary_mask(case.k_pool)
    assert not bool(cm[0, int(bad[0])].all())


# ----------------------------------------------------------------------------- batched

def test_batched_matches_single_windows():
    from synthetic.device import build_case
    import paper_2609_30884_amd as crf
    base = syn.WORKLOADS["qwen15b_mixed8"]
    items = [syn.Window(300, 3, 2), syn.Window(513, 26, 2), syn.Window(64, 0, 1)]
    # one set of base weights for every layer any item touches
    layers = sorted({l for w in items for l in range(w.l0, w.l0 + w.h)})
    cases = [build_case(base, 7, window=w, item=i, layers=layers) for i, w in enumerate(items)]
    for c in cases[1:]:   # share base weights (same model), keep per-item adapters
        c.weights_dev = cases[0].weights_dev
        c.weights = cases[0].weights
    cd = cdims(base.dims)
    ctx = crf.Context(cd, max(w.n_tokens for w in items), base.lora_rank)
    its, keep = [], []
    for c in cases:
        la = crf.lora_array(c.lora_dev, base.dims.n_layers)
        keep.append(la)
        kv = crf.kv_cache(c.k_pool, c.v_pool, c.block_table_dev, c.window.n_tokens, base.page_size)
        its.append(crf.window_item(c.hidden_dev, la, c.window.l0, c.window.h, kv, c.hidden_out))
    crf.recompute_window_batched(ctx, cd, crf.layer_weights_array(cases[0].weights_dev), its)
    torch.cuda.synchronize()
    for i, c in enumerate(cases):
        out, kv = oracle_window(c)
        assert_window_parity(c, out, kv, label=f"batched item {i}")


def test_batched_validates_every_item_first():
    from synthetic.device import build_case
    import paper_2609_30884_amd as crf
    base = syn.WORKLOADS["qwen15b_mixed8"]
    c = build_case(base, 7, window=syn.Window(128, 2, 1))
    cd = cdims(base.dims)
    ctx = crf.Context(cd, 128, base.lora_rank)
    la = crf.lora_array(c.lora_dev, base.dims.n_layers)
    kv = crf.kv_cache(c.k_pool, c.v_pool, c.block_table_dev, 128, base.page_size)
    good = crf.window_item(c.hidden_dev, la, 2, 1, kv, c.hidden_out)
    bad = crf.window_item(c.hidden_dev, la, 27, 2, kv, c.hidden_out)
    with pytest.raises(crf.CrfError) as ei:
        crf.recompute_window_batched(ctx, cd, crf.layer_weights_array(c.weights_dev), [good, bad])
    assert ei.value.status == 3 and "outside" in str(ei.value)
    torch.cuda.synchronize()
    from synthetic.device import canary_mask
    assert bool(canary_mask(c.k_pool).all()), "nothing may run when any item is invalid"


def _batched_cases(windows, seed=7):
    from synthetic.device import build_case
    base = syn.WORKLOADS["qwen15b_mixed8"]
    layers = sorted({l for w in windows for l in range(w.l0, w.l0 + w.h)})
    cases = [build_case(base, seed, window=w, item=i, layers=layers) for i, w in enumerate(windows)]
    for c in cases[1:]:
        c.weights_dev = cases[0].weights_dev
        c.weights = cases[0].weights
    return base, cases


def test_batched_lanes_match_in_order_run():
    """Independent items run on two lanes with timing off and in order with
    timing on: outputs and pages bitwise the same."""
    import paper_2609_30884_amd as crf
    from synthetic.device import canary_fill
    base, cases = _batched_cases([syn.Window(700, 3, 2), syn.Window(257, 26, 2), syn.Window(1030, 10, 1),
                                  syn.Window(64, 0, 3), syn.Window(1, 5, 1)])
    cd = cdims(base.dims)
    ctx = crf.Context(cd, max(c.window.n_tokens for c in cases), base.lora_rank)
    keep, its = [], []
    for c in cases:
        la = crf.lora_array(c.lora_dev, base.dims.n_layers)
        keep.append(la)
        kv = crf.kv_cache(c.k_pool, c.v_pool, c.block_table_dev, c.window.n_tokens, base.page_size)
        its.append(crf.window_item(c.hidden_dev, la, c.window.l0, c.window.h, kv, c.hidden_out))
    w = crf.layer_weights_array(cases[0].weights_dev)
    print("[case] batched lanes vs in-order", flush=True)
    ctx.set_timing(True)
    crf.recompute_window_batched(ctx, cd, w, its)
    torch.cuda.synchronize()
    ctx.set_timing(False)
    ctx.read_timing()
    ref = [(c.hidden_out.clone(), c.k_pool.clone(), c.v_pool.clone()) for c in cases]
    for c in cases:
        canary_fill(c.k_pool)
        canary_fill(c.v_pool)
        c.hidden_out.zero_()
    for _ in range(2):  # the second call reuses the lanes made by the first
        crf.recompute_window_batched(ctx, cd, w, its)
    torch.cuda.synchronize()
    assert ctx.device_errors() == 0
    for c, (h, k, v) in zip(cases, ref):
        assert bits_equal(c.hidden_out, h) and bits_equal(c.k_pool, k) and bits_equal(c.v_pool, v)


def test_batched_chained_items_run_in_order():
    """An item whose boundary state is another item's output is not
    independent: the batch runs in order and the second item sees the first
    one's output."""
    import paper_2609_30884_amd as crf
    base, cases = _batched_cases([syn.Window(300, 2, 1), syn.Window(300, 3, 1)])
    cd = cdims(base.dims)
    ctx = crf.Context(cd, 300, base.lora_rank)
    las = [crf.lora_array(c.lora_dev, base.dims.n_layers) for c in cases]
    kvs = [crf.kv_cache(c.k_pool, c.v_pool, c.block_table_dev, 300, base.page_size) for c in cases]
    mid = torch.empty_like(cases[0].hidden_out)
    its = [crf.window_item(cases[0].hidden_dev, las[0], 2, 1, kvs[0], mid),
           crf.window_item(mid, las[1], 3, 1, kvs[1], cases[1].hidden_out)]
    w = crf.layer_weights_array(cases[0].weights_dev)
    print("[case] batched chained items", flush=True)
    crf.recompute_window_batched(ctx, cd, w, its)
    torch.cuda.synchronize()
    got = cases[1].hidden_out.clone()
    # the same two windows as separate calls, in order
    mid2 = torch.empty_like(mid)
    crf.recompute_window(ctx, cd, cases[0].hidden_dev, w, las[0], 2, 1, kvs[0], mid2)
    crf.recompute_window(ctx, cd, mid2, w, las[1], 3, 1, kvs[1], cases[1].hidden_out)
    torch.cuda.synchronize()
    assert bits_equal(mid, mid2) and bits_equal(got, cases[1].hidden_out)


def _run_pair(crf, ctx, cd, w, its, batched):
    if batched:
        crf.recompute_window_batched(ctx, cd, w, its)
    else:
        for it in its:
            crf.recompute_window(ctx, cd, it.hidden_at_boundary, w, it.lora, it.l0, it.h, it.kv, it.hidden_out)
    torch.cuda.synchronize()


def test_batched_overlapping_views_run_in_order():
    """Items that share memory through different views (no base pointer in
    common) are not independent: (a) the second item's pools are the first's
    shifted by one layer, so their windows [2, 4) and [1, 3) write the same two
    layers; (b) the second item's boundary state starts 64 rows into the first
    one's output.  Each batch must equal the two windows run in order,
    bitwise."""
    import paper_2609_30884_amd as crf
    from synthetic.device import canary_fill
    n = 300
    base, cases = _batched_cases([syn.Window(n, 2, 2), syn.Window(n, 1, 2)])
    cd = cdims(base.dims)
    ctx = crf.Context(cd, n, base.lora_rank)
    w = crf.layer_weights_array(cases[0].weights_dev)
    las = [crf.lora_array(c.lora_dev, base.dims.n_layers) for c in cases]
    a, b = cases
    assert a.n_phys == b.n_phys
    shape = (base.dims.n_layers + 1,) + tuple(a.k_pool.shape[1:])
    kp = torch.empty(shape, dtype=a.k_pool.dtype, device="cuda")
    vp = torch.empty_like(kp)

    def pool_items():
        canary_fill(kp)
        canary_fill(vp)
        kva = crf.kv_cache(kp[:-1], vp[:-1], a.block_table_dev, n, base.page_size)
        kvb = crf.kv_cache(kp[1:], vp[1:], b.block_table_dev, n, base.page_size)
        return [crf.window_item(a.hidden_dev, las[0], 2, 2, kva, a.hidden_out),
                crf.window_item(b.hidden_dev, las[1], 1, 2, kvb, b.hidden_out)]

    print("[case] batched items on layer-shifted views of one pool", flush=True)
    _run_pair(crf, ctx, cd, w, pool_items(), batched=False)
    ref = (kp.clone(), vp.clone(), b.hidden_out.clone())
    _run_pair(crf, ctx, cd, w, pool_items(), batched=True)
    assert ctx.device_errors() == 0
    assert bits_equal(kp, ref[0]) and bits_equal(vp, ref[1]) and bits_equal(b.hidden_out, ref[2])

    # (b) hidden-state overlap: b's boundary = rows [64, 64 + n) of a buffer whose rows [0, n) are a's output
    buf = torch.empty((n + 64, base.dims.d_model), dtype=a.hidden_dev.dtype, device="cuda")

    def hidden_items():
        buf.zero_()
        buf[n:] = b.hidden_dev[n - 64:]
        canary_fill(a.k_pool)
        canary_fill(b.k_pool)
        canary_fill(a.v_pool)
        canary_fill(b.v_pool)
        kva = crf.kv_cache(a.k_pool, a.v_pool, a.block_table_dev, n, base.page_size)
        kvb = crf.kv_cache(b.k_pool, b.v_pool, b.block_table_dev, n, base.page_size)
        return [crf.window_item(a.hidden_dev, las[0], 2, 2, kva, buf[:n]),
                crf.window_item(buf[64:], las[1], 1, 2, kvb, b.hidden_out)]

    print("[case] batched item reading an overlapping part of another's output", flush=True)
    _run_pair(crf, ctx, cd, w, hidden_items(), batched=False)
    ref = (buf.clone(), b.k_pool.clone(), b.v_pool.clone(), b.hidden_out.clone())
    _run_pair(crf, ctx, cd, w, hidden_items(), batched=True)
    assert ctx.device_errors() == 0
    assert (bits_equal(buf, ref[0]) and bits_equal(b.k_pool, ref[1]) and bits_equal(b.v_pool, ref[2])
            and bits_equal(b.hidden_out, ref[3]))
