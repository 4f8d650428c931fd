"""First decoding step over a (hybrid) cached prefix on the GPU against the
oracle (Sec. 3.2 "Tail Influence"): logits of the last new token and the new
tokens' K/V written after the prefix, for caches whose layers before b come
from the current adapter and from b on from an older one."""
import numpy as np
import pytest

import synthetic as syn
from tests.helpers import TOL, TOL_ELEM, cdims, rel_to_rms, rms_rel

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

SMALL = dict(n_layers=4, d_model=768, n_q_heads=12, n_kv_heads=2, head_dim=64, d_ffn=2048)
VOCAB = 1024


def _setup(seed, n, m, base="qwen15b_4k", shape=SMALL, vocab=VOCAB, page_size=None):
    import dataclasses
    from oracle import oracle as O
    from synthetic.device import build_case, scatter_kv, to_dev
    wl = syn.WORKLOADS[base].with_dims(**shape).with_window(n_tokens=n + m, l0=0, h=shape["n_layers"])
    if page_size is not None:
        wl = dataclasses.replace(wl, page_size=page_size)
    dims = wl.dims
    N = dims.n_layers
    case = build_case(wl, seed, lora_version=3, layers=range(N))         # current adapter: version 3
    emb = syn.gen_hidden(wl, seed, n)
    x_new = syn.gen_new_tokens(wl, seed, m)
    lo_old = {l: syn.gen_lora_layer(wl, seed, l, 0) for l in range(N)}
    _, fresh, _ = O.prefill(emb, case.weights, case.lora, dims, wl.lora_scale)
    _, stale, _ = O.prefill(emb, case.weights, lo_old, dims, wl.lora_scale)
    r = syn.round_bf16
    fresh = {l: (r(k.astype(np.float32)), r(v.astype(np.float32))) for l, (k, v) in fresh.items()}
    stale = {l: (r(k.astype(np.float32)), r(v.astype(np.float32))) for l, (k, v) in stale.items()}
    g, head = syn.gen_head(wl, seed, vocab)
    dev = dict(x=to_dev(x_new, dims), g=to_dev(g, dims), head=to_dev(head, dims),
               logits=torch.empty(vocab, dtype=torch.float32, device="cuda"))
    return wl, case, x_new, fresh, stale, g, head, dev, scatter_kv


@pytest.mark.parametrize("b", [0, 2, 4])
def test_decode_logits_over_hybrid_cache(b):
    _check_decode(7, 300, 3, b)


# Longer prefixes split attention over the keys (the query heads of a KV group
# stacked on one tile's rows when they fit, else one workgroup per query
# head), split the LoRA down-projections over K, and run the projections with
# 4, 8 or 16 waves per workgroup.
SPLIT_CASES = {
    # 16 rows x 6 heads stacked; the last key split starts after the first 4
    # rows' positions (1020..1023), so those rows see no key in it
    "stacked_hd64": ("qwen7b_16k", dict(n_layers=2, d_model=1536, n_q_heads=12, n_kv_heads=2, head_dim=64,
                                        d_ffn=2048), 1020, 16, 1024),
    # one row, hd 128; gate/up on 8 waves, LM head on 4
    "one_row_hd128": ("qwen7b_16k", dict(n_layers=2, d_model=1024, n_q_heads=8, n_kv_heads=2, head_dim=128,
                                         d_ffn=8192), 700, 1, 16384),
    # 16 rows x 12 heads do not fit one tile: one workgroup per query head
    "per_head_hd128": ("qwen15b_4k", dict(n_layers=2, d_model=1536, n_q_heads=12, n_kv_heads=1, head_dim=128,
                                          d_ffn=2048), 600, 16, 1024),
    # d_ffn = 33 x 64: the down projection's 66 k-steps leave a partial last
    # batch of k-steps in the projection and LoRA kernels
    "ragged_ffn": ("qwen7b_16k", dict(n_layers=2, d_model=768, n_q_heads=12, n_kv_heads=2, head_dim=64,
                                      d_ffn=2112), 500, 4, 1024),
}


@pytest.mark.parametrize("name", list(SPLIT_CASES))
def test_decode_key_split_shapes(name):
    base, shape, n, m, vocab = SPLIT_CASES[name]
    _check_decode(11, n, m, 1, base=base, shape=shape, vocab=vocab)


# More than 16 new tokens take the window kernels with a position offset: the
# projection epilogue rotates and pages row r at position n + r, and attention
# runs query blocks at that offset over the prefix and the rows before them.
MANY_CASES = {
    "m40": (300, 40, None),
    "m257": (500, 257, None),
    # one-token pages: the page bases of a 2600-token prefix exceed what a
    # workgroup stages at once (key-split attention refills them mid-range)
    "m3_pages1": (2600, 3, 1),
    "m40_pages1": (2300, 40, 1),
}


@pytest.mark.parametrize("name", list(MANY_CASES))
def test_decode_many_new_tokens_and_page_refill(name):
    n, m, ps = MANY_CASES[name]
    _check_decode(13, n, m, 2, page_size=ps)


def _check_decode(seed, n, m, b, **kw):
    import paper_2609_30884_amd as crf
    from oracle import oracle as O
    from synthetic.device import gather_kv
    wl, case, x_new, fresh, stale, g, head, dev, scatter_kv = _setup(seed, n, m, **kw)
    dims, N = wl.dims, wl.dims.n_layers
    hyb = O.hybrid_caches(fresh, stale, b, N)
    for l in range(N):
        scatter_kv(case.k_pool, l, case.block_table, wl.page_size, hyb[l][0])
        scatter_kv(case.v_pool, l, case.block_table, wl.page_size, hyb[l][1])
    print(f"[case] decode n={n} m={m} boundary b={b} dims={dims}", flush=True)
    cd = cdims(dims)
    ctx = crf.Context(cd, n + m, wl.lora_rank)
    kv = crf.kv_cache(case.k_pool, case.v_pool, case.block_table_dev, n, wl.page_size)
    crf.decode_logits(ctx, cd, dev["x"], crf.layer_weights_array(case.weights_dev),
                      crf.lora_array(case.lora_dev, N), kv, dev["g"], dev["head"], dev["logits"])
    torch.cuda.synchronize()
    assert ctx.device_errors() == 0
    z_gpu = dev["logits"].cpu().numpy().astype(np.float64)
    z_ref = O.decode_logits(x_new, hyb, case.weights, case.lora, dims, g, head, wl.lora_scale)
    errs = {"logits": (rms_rel(z_gpu, z_ref), rel_to_rms(z_gpu, z_ref))}
    # the new tokens' K/V after the prefix, layer by layer
    h = x_new
    rows = np.arange(n, n + m)
    for l in range(N):
        h, k, v = O.decode_layer(h, hyb[l][0], hyb[l][1], case.weights[l], case.lora[l], dims, wl.lora_scale)
        kg = gather_kv(case.k_pool, l, case.block_table, n + m, wl.page_size, rows)
        vg = gather_kv(case.v_pool, l, case.block_table, n + m, wl.page_size, rows)
        errs[f"Knew{l}"] = (rms_rel(kg, k), rel_to_rms(kg, k))
        errs[f"Vnew{l}"] = (rms_rel(vg, v), rel_to_rms(vg, v))
    print("[parity] decode " + " ".join(f"{k}=({a:.2e},{e:.2e})" for k, (a, e) in errs.items()), flush=True)
    bad = {k: v for k, v in errs.items() if not (v[0] <= TOL["bf16"] and v[1] <= TOL_ELEM["bf16"])}
    assert not bad, bad
    # the prefix slots keep the planted cache
    for l in range(N):
        kp = gather_kv(case.k_pool, l, case.block_table, n, wl.page_size)
        assert np.array_equal(kp.astype(np.float32), hyb[l][0].astype(np.float32))


def test_decode_rejects_unsupported_requests():
    import dataclasses
    import paper_2609_30884_amd as crf
    seed, n, m = 7, 64, 2
    wl, case, x_new, fresh, stale, g, head, dev, _ = _setup(seed, n, m)
    cd = cdims(wl.dims)
    ctx = crf.Context(cd, n + m, wl.lora_rank)
    kv = crf.kv_cache(case.k_pool, case.v_pool, case.block_table_dev, n, wl.page_size)
    args = (crf.layer_weights_array(case.weights_dev), crf.lora_array(case.lora_dev, wl.dims.n_layers), kv)
    with pytest.raises(crf.CrfError) as ei:         # vocab not a multiple of 8
        crf.decode_logits(ctx, cd, dev["x"], *args, dev["g"], dev["head"][:1020], dev["logits"])
    assert ei.value.status == 4
    small = crf.Context(cd, n, wl.lora_rank)         # prefix + new tokens exceed max_tokens
    with pytest.raises(crf.CrfError) as ei:
        crf.decode_logits(small, cd, dev["x"], *args, dev["g"], dev["head"], dev["logits"])
    assert ei.value.status == 5
    wl32 = dataclasses.replace(syn.WORKLOADS["tiny_f32"])
    cd32 = cdims(wl32.dims)
    ctx32 = crf.Context(cd32, 16, 8)
    with pytest.raises(crf.CrfError) as ei:          # fp32 contexts: unsupported
        crf.decode_logits(ctx32, cd32, dev["x"], *args, dev["g"], dev["head"], dev["logits"])
    assert ei.value.status in (1, 4)
