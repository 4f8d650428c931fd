"""Host-side pieces of the benchmark: a stored HBM-traffic figure is reported
only while the kernel sources it was measured on are unchanged."""
import importlib.util
import json
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("crf_bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_traffic_follows_the_kernel_sources(tmp_path, monkeypatch):
    bench = _bench()
    prof = tmp_path / "profiles"
    prof.mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    rec = {"bytes_per_launch": 123, "sources_sha256": bench.kernel_sources_digest("gemm_gateup")}
    (prof / "traffic_gemm_gateup_w.json").write_text(json.dumps(rec))
    assert bench.stored_traffic("gemm_gateup", "w") == 123
    rec["sources_sha256"] = "0" * 64
    (prof / "traffic_gemm_gateup_w.json").write_text(json.dumps(rec))
    assert bench.stored_traffic("gemm_gateup", "w") is None
    del rec["sources_sha256"]
    (prof / "traffic_gemm_gateup_w.json").write_text(json.dumps(rec))
    assert bench.stored_traffic("gemm_gateup", "w") is None
    assert bench.stored_traffic("gemm_gateup", "missing") is None


def test_digest_covers_each_family():
    bench = _bench()
    g, a = bench.kernel_sources_digest("gemm_down"), bench.kernel_sources_digest("attn")
    assert g and a and g != a
    assert bench.kernel_sources_digest("gemm_qkv") == g
    assert bench.kernel_sources_digest("norm") is None


def test_work_accounting_matches_brute_force_counts():
    """The roofline numerators: per-kernel FLOP and window FLOP against counts
    made by enumeration on a tiny shape (every multiply-add of each projection,
    its LoRA up-projection, and one 2*hd-FLOP product per (query head, query,
    visible key) for scores and again for P.V, keys at or before the query)."""
    import synthetic as syn
    bench = _bench()
    dims = syn.Dims(n_layers=2, d_model=64, n_q_heads=4, n_kv_heads=2, head_dim=16, d_ffn=96)
    n, r = 7, 3
    targets = syn.TARGETS
    macs = {t: dims.target_shape(t)[0] * dims.target_shape(t)[1] for t in targets}
    pairs = sum(1 for q in range(n) for p in range(n) if p <= q)
    up = {t: r * dims.target_shape(t)[0] for t in targets}
    down = {t: r * dims.target_shape(t)[1] for t in targets}
    want = {
        "gemm_qkv": 2 * n * sum(macs[t] + up[t] for t in "qkv"),
        "gemm_o": 2 * n * (macs["o"] + up["o"]),
        "gemm_gateup": 2 * n * sum(macs[t] + up[t] for t in ("gate", "up")),
        "gemm_down": 2 * n * (macs["down"] + up["down"]),
        "attn": dims.n_q_heads * pairs * 2 * (2 * dims.head_dim),
    }
    assert bench.kernel_flops(dims, n, r, targets) == want
    total, parts = bench.window_flops(dims, n, 2, r, targets)
    # the window adds the LoRA down-projections (their own passes) to the kernels' work, per layer
    assert total == 2 * (sum(want.values()) + 2 * n * sum(down.values()))
    assert parts["attn"] == want["attn"]
    # no adapter: the projections alone
    assert bench.kernel_flops(dims, n, r, ())["gemm_o"] == 2 * n * macs["o"]
