"""Degenerate and boundary cases of the bf16 path against the oracle:
prefix lengths around the 16-token page, the 64-key attention tile, the
128-query attention block and the 256-row GEMM tile (including n = 1, where
attention returns V[0]); an empty prefix; no adapter and a partial adapter;
and a prefix longer than the context's workspace."""
import dataclasses

import pytest

import synthetic as syn
from tests.helpers import assert_window_parity, bits_equal, cdims, oracle_window, run_gpu_window

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

SMALL = dict(n_layers=4, d_model=768, n_q_heads=12, n_kv_heads=2, head_dim=64, d_ffn=2048)


def _wl(kind, n, **kw):
    base = syn.WORKLOADS["qwen15b_4k"]
    if kind == "small":
        base = base.with_dims(**SMALL)
    wl = base.with_window(n_tokens=n, l0=1, h=2)
    return dataclasses.replace(wl, **kw) if kw else wl


@pytest.mark.parametrize("kind,n", [("small", n) for n in (1, 2, 15, 16, 17, 63, 64, 65, 127, 128, 129, 255, 256, 257)]
                         + [("qwen15b", n) for n in (1, 17, 129, 257)])
def test_bf16_boundary_lengths(kind, n):
    from synthetic.device import build_case
    print(f"[case] {kind} n={n}", flush=True)
    case = build_case(_wl(kind, n), 17)
    run_gpu_window(case)
    torch.cuda.synchronize()
    out, kv = oracle_window(case)
    assert_window_parity(case, out, kv, label=f"{kind} n={n}")


@pytest.mark.parametrize("targets", [(), ("q", "v"), syn.TARGETS])
def test_bf16_absent_and_partial_adapter(targets):
    from synthetic.device import build_case
    wl = _wl("small", 300, lora_targets=tuple(targets))
    print(f"[case] adapter targets {targets}", flush=True)
    case = build_case(wl, 29)
    run_gpu_window(case)
    torch.cuda.synchronize()
    out, kv = oracle_window(case)
    assert_window_parity(case, out, kv, label=f"targets={targets}")


def test_bf16_null_adapter_equals_empty_adapter():
    import paper_2609_30884_amd as crf
    from synthetic.device import build_case
    wl = _wl("small", 200, lora_targets=())
    case = build_case(wl, 7)
    ctx = run_gpu_window(case)
    torch.cuda.synchronize()
    k1, v1, h1 = case.k_pool.clone(), case.v_pool.clone(), case.hidden_out.clone()
    kv = crf.kv_cache(case.k_pool, case.v_pool, case.block_table_dev, 200, wl.page_size)
    crf.recompute_window(ctx, cdims(wl.dims), case.hidden_dev, crf.layer_weights_array(case.weights_dev), None,
                         1, 2, kv, case.hidden_out)
    torch.cuda.synchronize()
    assert bits_equal(case.k_pool, k1) and bits_equal(case.v_pool, v1) and bits_equal(case.hidden_out, h1)


def test_bf16_empty_prefix_is_noop():
    import paper_2609_30884_amd as crf
    from synthetic.device import build_case, canary_mask
    wl = _wl("small", 64)
    case = build_case(wl, 7)
    ctx = crf.Context(cdims(wl.dims), 64, wl.lora_rank)
    kv = crf.kv_cache(case.k_pool, case.v_pool, case.block_table_dev, 0, wl.page_size)
    case.hidden_out.zero_()
    crf.recompute_window(ctx, cdims(wl.dims), case.hidden_dev, crf.layer_weights_array(case.weights_dev),
                         crf.lora_array(case.lora_dev, wl.dims.n_layers), 1, 2, kv, case.hidden_out)
    torch.cuda.synchronize()
    assert bool(canary_mask(case.k_pool).all()) and bool(canary_mask(case.v_pool).all())
    assert bool((case.hidden_out == 0).all())
    assert ctx.device_errors() == 0


def test_prefix_longer_than_workspace_is_rejected():
    import paper_2609_30884_amd as crf
    from synthetic.device import build_case, canary_mask
    wl = _wl("small", 200)
    case = build_case(wl, 7)
    ctx = crf.Context(cdims(wl.dims), 100, wl.lora_rank)
    with pytest.raises(crf.CrfError) as ei:
        run_gpu_window(case, ctx=ctx)
    assert ei.value.status == 5
    torch.cuda.synchronize()
    assert bool(canary_mask(case.k_pool).all()), "nothing may run when the request is rejected"


@pytest.mark.parametrize("base,dims,n", [
    ("qwen15b_4k", dict(n_layers=4, d_model=768, n_q_heads=12, n_kv_heads=2, head_dim=64, d_ffn=2048), 5500),
    ("qwen15b_4k", dict(n_layers=4, d_model=768, n_q_heads=24, n_kv_heads=4, head_dim=128, d_ffn=1024), 2800),
    # adapters on all seven projections over 8200 tokens: the LoRA down-projections
    # take 64 tokens per workgroup (8 tokens in the last one)
    ("qwen7b_16k", dict(n_layers=4, d_model=256, n_q_heads=2, n_kv_heads=1, head_dim=128, d_ffn=512), 8200),
    # adapters on all seven projections, 22 token tiles x 16 gate/up tiles on 256
    # workgroups: 36 workgroups' items cross a token-tile group, so their fused
    # down-projection adapter sums are flushed as two runs
    ("qwen7b_16k", dict(n_layers=4, d_model=768, n_q_heads=12, n_kv_heads=2, head_dim=64, d_ffn=2048), 5500),
])
def test_bf16_longer_prefixes(base, dims, n):
    """Longer ragged prefixes (dozens of query blocks per head, more query
    heads than model width) with head_dim 64 and 128."""
    from synthetic.device import build_case
    wl = syn.WORKLOADS[base].with_dims(**dims).with_window(n_tokens=n, l0=1, h=2)
    print(f"[case] longer prefix {dims} n={n}", flush=True)
    case = build_case(wl, 29)
    run_gpu_window(case)
    torch.cuda.synchronize()
    out, kv = oracle_window(case)
    assert_window_parity(case, out, kv, label=f"longer prefix n={n}")


@pytest.mark.parametrize("rank,d_ffn", [(8, 2112), (16, 2112), (32, 2112)])
def test_bf16_adapter_ranks(rank, d_ffn):
    """Adapters on all seven projections at ranks below, at and above the
    16 that the gate/up epilogue's fused down-projection sums take (rank 32
    goes through the separate down-projection pass), with d_ffn = 33 x 64, so
    the last gate/up tile holds only gate/up rows of 64 features and its
    second feature half lies past d_ffn."""
    from synthetic.device import build_case
    base = syn.WORKLOADS["qwen7b_16k"].with_dims(n_layers=4, d_model=768, n_q_heads=12, n_kv_heads=2, head_dim=64,
                                                  d_ffn=d_ffn)
    wl = dataclasses.replace(base.with_window(n_tokens=700, l0=1, h=2), lora_rank=rank)
    print(f"[case] adapter rank {rank} d_ffn {d_ffn} n=700", flush=True)
    case = build_case(wl, 31)
    run_gpu_window(case)
    torch.cuda.synchronize()
    out, kv = oracle_window(case)
    assert_window_parity(case, out, kv, label=f"rank {rank} d_ffn {d_ffn}")


@pytest.mark.parametrize("kind,h", [("small", 1), ("small", 2), ("f32", 2)])
def test_hidden_out_may_alias_the_boundary_state(kind, h):
    """hidden_out on the same buffer as hidden_at_boundary gives bitwise the
    output and pages of a run into a separate buffer."""
    import paper_2609_30884_amd as crf
    from synthetic.device import build_case, canary_fill
    if kind == "f32":
        wl = syn.WORKLOADS["tiny_f32"].with_window(n_tokens=150, l0=1, h=h)
    else:
        wl = _wl("small", 300)
        wl = wl.with_window(l0=1, h=h)
    print(f"[case] aliasing {kind} h={h}", flush=True)
    case = build_case(wl, 5)
    run_gpu_window(case)
    torch.cuda.synchronize()
    out_sep = case.hidden_out.clone()
    k_sep, v_sep = case.k_pool.clone(), case.v_pool.clone()
    canary_fill(case.k_pool)
    canary_fill(case.v_pool)
    buf = case.hidden_dev.clone()
    cd = cdims(wl.dims)
    ctx = crf.Context(cd, wl.windows[0].n_tokens, wl.lora_rank)
    kv = crf.kv_cache(case.k_pool, case.v_pool, case.block_table_dev, wl.windows[0].n_tokens, wl.page_size)
    crf.recompute_window(ctx, cd, buf, crf.layer_weights_array(case.weights_dev),
                         crf.lora_array(case.lora_dev, wl.dims.n_layers), 1, h, kv, buf)
    torch.cuda.synchronize()
    assert bits_equal(buf, out_sep)
    assert bits_equal(case.k_pool, k_sep) and bits_equal(case.v_pool, v_sep)
