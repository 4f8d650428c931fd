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
