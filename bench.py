"""Benchmark: bounded KV-window recomputation on one MI355X.

One step = one crf_recompute_window call over the 7B-shaped workload: 16384
prefix tokens re-run through decoder layers [14, 16) (Qwen2.5-7B shapes,
rank-16 LoRA on all seven projections, paged bf16 KV cache with 16-token
pages), inputs resident in HBM before the timed region.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

Other workloads (one JSON line each): tiny_f32, qwen15b_4k, qwen7b_16k_suffix
(the 24-layer affected suffix), qwen15b_mixed8 (8 ragged stale caches through
the batched call), drift (crf_layer_drift over 28 layers and 4 stored
adapter versions at 1.5B shapes), trajectory (maintenance over 32 adapter
updates: fresh, exact suffix, drift policy, reuse), tail (first-step logits
over hybrid caches at every boundary, timed decoding step) and copy (a 1 GiB
elementwise pass that calibrates the HBM byte counters).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_2609_30884_amd", "csrc")
# the sources each kernel family is built from: a stored HBM-traffic figure
# counts only while they are byte for byte the ones the counters ran on
TRAFFIC_SOURCES = {"gemm": ("gemm_bf16.hip", "common.hpp", "kernels.hpp"),
                   "attn": ("attn_bf16.hip", "common.hpp", "kernels.hpp")}


def kernel_sources_digest(kernel: str) -> str | None:
    files = TRAFFIC_SOURCES.get(kernel.split("_")[0])
    if not files:
        return None
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def stored_traffic(kernel: str, workload: str):
    """HBM bytes per launch from profiles/traffic_<kernel>_<workload>.json
    (copy-calibrated FETCH_SIZE + WRITE_SIZE), or None when there is none or
    the kernel's sources have changed since the counters were taken."""
    prof = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    try:
        rec = json.load(open(prof))
    except (OSError, ValueError):
        return None
    if rec.get("sources_sha256") != kernel_sources_digest(kernel):
        return None
    return rec.get("bytes_per_launch")
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "recomputed token-layers/sec and ms per 16K-token window (7B-shape); MFMA util"
SHAPE_NAME = {3584: "Qwen2.5-7B", 1536: "Qwen2.5-1.5B"}
PROFILE_STEPS = 3       # untimed steps with every kernel class under event timing
PEAK_BF16 = 2.5e15      # MI355X dense bf16 MFMA, FLOP/s
PEAK_F32_VALU = 157.3e12  # MI355X fp32 vector FLOP/s (the fp32 path runs on plain FMAs)
PEAK_HBM = 8.0e12       # bytes/s


def window_flops(dims, n, h, rank, targets):
    """Algorithmic FLOP of one window (causal attention counts only q <= p)."""
    d, dq, dkv, f = dims.d_model, dims.dq, dims.dkv, dims.d_ffn
    gemm = 2 * n * (d * (dq + 2 * dkv) + dq * d + d * 2 * f + f * d)
    lora = 0
    for t in targets:
        d_out, d_in = dims.target_shape(t)
        lora += 2 * n * rank * (d_in + d_out)
    attn = 2 * 2 * dims.n_q_heads * dims.head_dim * (n * (n + 1) // 2)
    return h * (gemm + lora + attn), {"gemm": gemm, "lora": lora, "attn": attn}


def kernel_flops(dims, n, rank, targets):
    """Algorithmic FLOP per launch of the projection kernels (base GEMM plus the
    in-kernel LoRA up-projection) and of the attention kernel."""
    d, dq, dkv, f = dims.d_model, dims.dq, dims.dkv, dims.d_ffn

    def up(ts):
        return sum(2 * n * rank * dims.target_shape(t)[0] for t in ts if t in targets)
    return {
        "gemm_qkv": 2 * n * d * (dq + 2 * dkv) + up(("q", "k", "v")),
        "gemm_o": 2 * n * dq * d + up(("o",)),
        "gemm_gateup": 2 * n * d * 2 * f + up(("gate", "up")),
        "gemm_down": 2 * n * f * d + up(("down",)),
        "attn": 2 * 2 * dims.n_q_heads * dims.head_dim * (n * (n + 1) // 2),
    }


def cpu_baseline(case, n_layers: int):
    """The oracle (fp64 numpy) over the whole prefix of the same window, for
    its first n_layers layers; returns token-layers/s, seconds, BLAS threads
    and the BLAS name."""
    import numpy as np
    from oracle import oracle as O
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        threads = max([i.get("num_threads", 1) for i in info] or [1])
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')}"
    except Exception:
        threads = len(os.sched_getaffinity(0))
    win = case.window
    t0 = time.perf_counter()
    O.recompute_window(case.hidden, case.weights, case.lora, win.l0, n_layers, case.dims, case.wl.lora_scale)
    dt = time.perf_counter() - t0
    return win.n_tokens * n_layers / dt, dt, threads, blas


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def tail_skipped_flops(dims, n, rank, targets):
    """Algorithmic FLOP the K/V-only last layer does not run: Q, attention, O
    and the MLP (with their adapter deltas)."""
    d, dq, f = dims.d_model, dims.dq, dims.d_ffn
    gemm = 2 * n * (d * dq + dq * d + d * 2 * f + f * d)
    lora = sum(2 * n * rank * sum(dims.target_shape(t)) for t in targets if t in ("q", "o", "gate", "up", "down"))
    attn = 2 * 2 * dims.n_q_heads * dims.head_dim * (n * (n + 1) // 2)
    return gemm + lora + attn


def hbm_bytes(dims, n, h, rank, targets, kv_tail):
    """Algorithmic HBM bytes per window of the HBM-bound kernel classes (each
    tensor read or written once): RMSNorm (bf16 or fp32 residual in, bf16 out;
    the window's first norm of a few rows also writes the fp32 residual copy,
    which longer windows read from the boundary state instead) and the skinny
    LoRA-down passes (activation in, rank columns out)."""
    d, dq, f = dims.d_model, dims.dq, dims.d_ffn
    first = n * d * (2 + 2) if n > 16 else n * d * (2 + 4 + 2)
    norm = first + (2 * h - 1 - (1 if kv_tail else 0)) * n * d * (4 + 2)
    r3 = 3 * rank * 2
    per_layer = {"qkv": n * d * 2 + n * r3, "o": n * dq * 2 + n * r3, "gateup": n * d * 2 + n * r3,
                 "down": n * f * 2 + n * r3}
    has = {"qkv": any(t in targets for t in "qkv"), "o": "o" in targets,
           "gateup": "gate" in targets or "up" in targets, "down": "down" in targets}
    full = sum(v for k, v in per_layer.items() if has[k])
    tail = (per_layer["qkv"] if has["qkv"] else 0) if kv_tail else full
    return {"norm": norm, "lora_down": (h - 1) * full + tail}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen7b_16k")
    ap.add_argument("--seed", type=int, default=7)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-layers", type=int, default=1,
                    help="window layers the CPU oracle runs over the whole prefix (bounded CPU time)")
    ap.add_argument("--updates", type=int, default=32, help="trajectory workload: number of adapter updates")
    ap.add_argument("--restart-every", type=int, default=1,
                    help="trajectory workload: retained boundary states every k layers (windows run as one call "
                         "per span between them)")
    ap.add_argument("--no-hidden-out", action="store_true",
                    help="window without hidden_out: the last layer runs its K/V projections only")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the recomputation path is built and measured on a single MI355X "
              f"(--gpus {args.gpus} is not supported: no part of it is sharded over GPUs).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_30884_amd as crf
    import synthetic as syn
    from synthetic.device import build_case

    crf.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    device = crf.device_info(0)
    if args.workload == "drift":
        return bench_drift(args)
    if args.workload == "qwen15b_mixed8":
        return bench_mixed(args)
    if args.workload == "copy":
        return bench_copy(args)
    if args.workload == "trajectory":
        return bench_trajectory(args)
    if args.workload == "tail":
        return bench_tail(args)
    wl = syn.WORKLOADS[args.workload]
    dims = wl.dims
    win = wl.window
    keep_host = not args.no_cpu_baseline
    t_gen = time.perf_counter()
    case = build_case(wl, args.seed, keep_host=keep_host)
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t_gen
    print(f"[bench] inputs ready in {t_gen:.1f}s: {wl.name} n={win.n_tokens} window=[{win.l0},{win.l0 + win.h})",
          file=sys.stderr, flush=True)

    cd = crf.make_dims(dims.n_layers, dims.d_model, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.d_ffn,
                       dims.rms_eps, dims.rope_theta, dims.dtype)
    ctx = crf.Context(cd, win.n_tokens, wl.lora_rank)
    weights = crf.layer_weights_array(case.weights_dev)
    lora = crf.lora_array(case.lora_dev, dims.n_layers)
    kv = crf.kv_cache(case.k_pool, case.v_pool, case.block_table_dev, win.n_tokens, wl.page_size)
    stream = torch.cuda.current_stream()

    hout = None if args.no_hidden_out else case.hidden_out

    def step():
        crf.recompute_window(ctx, cd, case.hidden_dev, weights, lora, win.l0, win.h, kv, hout, stream)

    kflops = kernel_flops(dims, win.n_tokens, wl.lora_rank, wl.lora_targets)
    if args.no_hidden_out:
        kflops.pop("gemm_qkv")   # the tail layer's launch is K/V-only: launches differ in size
    for _ in range(args.warmup):
        step()
    # per-kernel-class times from PROFILE_STEPS untimed steps with every class
    # bracketed by events; the timed region then brackets only the dominant
    # class (each bracketed launch adds two event records to the stream)
    prof_steps = min(PROFILE_STEPS, max(args.steps, 1))
    torch.cuda.synchronize()
    ctx.set_timing(True)
    ctx.read_timing()
    for _ in range(prof_steps):
        step()
    torch.cuda.synchronize()
    ctx.set_timing(False)
    timing = ctx.read_timing()
    dom = max((k for k in timing if k in kflops and timing[k][1]), key=lambda k: timing[k][0])
    ctx.set_timing(True, classes=[dom])
    ctx.read_timing()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ctx.set_timing(False)
    dom_timing = ctx.read_timing()[dom]
    flags = ctx.device_errors()
    assert flags == 0, f"device error flags {flags}"

    ms = 1e3 * elapsed / args.steps
    tl_per_s = win.n_tokens * win.h * args.steps / elapsed
    f_win, f_parts = window_flops(dims, win.n_tokens, win.h, wl.lora_rank, wl.lora_targets)
    if args.no_hidden_out:
        f_win -= tail_skipped_flops(dims, win.n_tokens, wl.lora_rank, wl.lora_targets)
    hbm = hbm_bytes(dims, win.n_tokens, win.h, wl.lora_rank, wl.lora_targets, args.no_hidden_out)
    kernels = {}
    for k, (tot_ms, cnt) in timing.items():
        if cnt:
            avg = tot_ms / cnt
            e = {"avg_ms": round(avg, 4), "launches": cnt, "share": round(tot_ms / (ms * prof_steps), 4)}
            if k in kflops:
                e["tflops"] = round(kflops[k] / (avg * 1e-3) / 1e12, 1)
            if k in hbm:
                e["gbps"] = round(hbm[k] * prof_steps / (tot_ms * 1e-3) / 1e9, 1)
            kernels[k] = e
    # the roofline's kernel time: its launches inside the timed region
    dom_avg_s = dom_timing[0] / dom_timing[1] * 1e-3
    kernels[dom]["avg_ms_timed"] = round(dom_avg_s * 1e3, 4)
    achieved = kflops[dom] / dom_avg_s
    peak = PEAK_BF16 if dims.dtype == "bf16" else PEAK_F32_VALU
    traffic = stored_traffic(dom, wl.name)

    out = {
        "metric": METRIC,
        "value": round(tl_per_s, 1),
        "unit": "token-layers/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if dims.dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1) boundary state, random-init N(0,0.02) weights, LoRA A~N(0,1/8), "
                "B~N(0,0.01)+N(0,0.005)); no dataset or checkpoint",
        "config": {
            "workload": f"{wl.name}: {SHAPE_NAME.get(dims.d_model, 'synthetic')}-shaped bounded window, "
                        f"{win.n_tokens}-token prefix, layers "
                        f"[{win.l0},{win.l0 + win.h}) of {dims.n_layers}, LoRA rank {wl.lora_rank} on "
                        f"{','.join(wl.lora_targets)}, paged KV {wl.page_size}-token pages"
                        + (", no hidden output (K/V-only last layer)" if args.no_hidden_out else ""),
            "n_tokens": win.n_tokens, "l0": win.l0, "h": win.h, "d_model": dims.d_model, "n_q_heads": dims.n_q_heads,
            "n_kv_heads": dims.n_kv_heads, "head_dim": dims.head_dim, "d_ffn": dims.d_ffn, "lora_rank": wl.lora_rank,
        },
        "mfma_util": round(f_win / (elapsed / args.steps) / peak, 4),
        "window_tflops": round(f_win / (elapsed / args.steps) / 1e12, 1),
        "roofline": {"bound": "mfma" if dims.dtype == "bf16" else "alu", "kernel": dom,
                     "achieved": round(achieved / 1e12, 1), "peak": round(peak / 1e12, 1), "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": traffic},
        "kernels": kernels,
        "device": device,
    }
    if not args.no_cpu_baseline:
        nl = max(1, min(args.cpu_sample_layers, win.h))
        print(f"[bench] cpu baseline: oracle over {win.n_tokens} tokens, {nl} layer(s) ...", file=sys.stderr,
              flush=True)
        v, dt, thr, blas = cpu_baseline(case, nl)
        layers = f"layer {win.l0}" if nl == 1 else f"layers [{win.l0},{win.l0 + nl})"
        out["cpu_baseline"] = {
            "value": round(v, 1), "unit": "token-layers/s", "cores": thr, "kind": "oracle",
            "sample": f"fp64 numpy oracle, {layers} of the window [{win.l0},{win.l0 + win.h}) over all "
                      f"{win.n_tokens} of {win.n_tokens} prefix tokens (full causal attention; {dt:.1f} s)",
            "cpu": cpu_model(), "blas": blas,
        }
    print(json.dumps(out), flush=True)


def _timed(step, steps, warmup, ctx=None, events_in_timed=False):
    """Wall time of `steps` steps after `warmup` untimed ones.  With a
    context, per-kernel-class times come from PROFILE_STEPS further untimed
    steps with event timing on, and the timed region runs without events; with
    events_in_timed they come from the timed region itself."""
    import torch
    for _ in range(warmup):
        step()
    timing = None
    if ctx is not None and events_in_timed:
        torch.cuda.synchronize()
        ctx.set_timing(True)
        ctx.read_timing()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        ctx.set_timing(False)
        return elapsed, ctx.read_timing()
    if ctx is not None:
        torch.cuda.synchronize()
        ctx.set_timing(True)
        ctx.read_timing()
        for _ in range(min(PROFILE_STEPS, max(steps, 1))):
            step()
        torch.cuda.synchronize()
        ctx.set_timing(False)
        timing = ctx.read_timing()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    return elapsed, timing


def bench_mixed(args):
    """8 independent stale caches (1.5B shapes, ragged n, own l0/h/adapter) in one
    crf_recompute_window_batched call per step."""
    import torch
    import paper_2609_30884_amd as crf
    import synthetic as syn
    from synthetic.device import build_case
    wl = syn.WORKLOADS["qwen15b_mixed8"]
    dims = wl.dims
    layers = sorted({l for w in wl.windows for l in range(w.l0, w.l0 + w.h)})
    # one base model (weights of every layer any item touches), one adapter version per item
    cases = [build_case(wl, args.seed, window=w, item=i, layers=layers, keep_host=False, with_weights=(i == 0))
             for i, w in enumerate(wl.windows)]
    cd = crf.make_dims(dims.n_layers, dims.d_model, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.d_ffn,
                       dims.rms_eps, dims.rope_theta, dims.dtype)
    ctx = crf.Context(cd, max(w.n_tokens for w in wl.windows), wl.lora_rank)
    weights = crf.layer_weights_array(cases[0].weights_dev)
    keep, items = [], []
    for c in cases:
        la = crf.lora_array(c.lora_dev, dims.n_layers)
        keep.append(la)
        kv = crf.kv_cache(c.k_pool, c.v_pool, c.block_table_dev, c.window.n_tokens, wl.page_size)
        items.append(crf.window_item(c.hidden_dev, la, c.window.l0, c.window.h, kv, c.hidden_out))
    stream = torch.cuda.current_stream()
    elapsed, timing = _timed(lambda: crf.recompute_window_batched(ctx, cd, weights, items, stream), args.steps,
                             args.warmup, ctx)
    tl = sum(w.n_tokens * w.h for w in wl.windows)
    f = sum(window_flops(dims, w.n_tokens, w.h, wl.lora_rank, wl.lora_targets)[0] for w in wl.windows)
    ms = 1e3 * elapsed / args.steps
    out = {
        "metric": METRIC, "value": round(tl * args.steps / elapsed, 1), "unit": "token-layers/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "qwen15b_mixed8: 8 stale caches, Qwen2.5-1.5B shapes, ragged n/l0/h, own LoRA "
                               "version each, one batched call",
                   "items": [[w.n_tokens, w.l0, w.h] for w in wl.windows]},
        "mfma_util": round(f / (elapsed / args.steps) / PEAK_BF16, 4),
        "kernels": {k: {"avg_ms": round(v[0] / v[1], 4), "launches": v[1]} for k, v in timing.items() if v[1]},
    }
    print(json.dumps(out), flush=True)


def bench_drift(args):
    """crf_layer_drift over 28 layers x 4 stored versions (1.5B shapes, rank 16 on q,k,v,o)."""
    import numpy as np
    import torch
    import paper_2609_30884_amd as crf
    import synthetic as syn
    from synthetic.device import lora_to_dev
    wl = syn.WORKLOADS["qwen15b_mixed8"]
    dims = wl.dims
    n_versions = 4
    states = [[lora_to_dev(syn.gen_lora_layer(wl, args.seed, l, v), wl.lora_rank, 1.0, dims)
               for l in range(dims.n_layers)] for v in range(n_versions + 1)]
    cd = crf.make_dims(dims.n_layers, dims.d_model, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.d_ffn,
                       dims.rms_eps, dims.rope_theta, dims.dtype)
    ctx = crf.Context(cd, 1, wl.lora_rank)
    cur = crf.lora_array(states[-1], dims.n_layers)
    vers = [crf.lora_array(s_, dims.n_layers) for s_ in states[:-1]]
    anchors = syn.gen_anchor_versions(dims.n_layers, n_versions, args.seed)
    sens = torch.from_numpy(syn.gen_sensitivity(dims.n_layers, args.seed)).cuda()
    drift = torch.empty(dims.n_layers, device="cuda")
    risk = torch.empty_like(drift)
    stream = torch.cuda.current_stream()
    elapsed, timing = _timed(lambda: crf.layer_drift(ctx, cd, cur, vers, anchors, sens, drift, risk, None,
                                                      stream=stream), args.steps, args.warmup, ctx,
                             events_in_timed=True)
    n_params = sum(int(a.numel() + b.numel()) for l in states[-1] for a, b in l["targets"].values())
    bytes_per_call = 2 * n_params * 2 * n_versions   # current + version, bf16, per version
    ms = 1e3 * elapsed / args.steps
    kern_ms = timing["drift"][0] / max(timing["drift"][1], 1) * 1e-3 * 2  # two kernels per call
    out = {
        "metric": "adapter drift scoring: ms per call over all layers and stored versions", "value": round(ms, 4),
        "unit": "ms", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"drift: {dims.n_layers} layers, {n_versions} stored versions, {n_params} adapter "
                               f"parameters per version"},
        "roofline": {"bound": "hbm", "achieved": round(bytes_per_call / (timing['drift'][0] / args.steps * 1e-3) / 1e9, 1),
                     "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                     "frac": round(bytes_per_call / (timing['drift'][0] / args.steps * 1e-3) / PEAK_HBM, 4),
                     "traffic": None},
        "kernels": {k: {"avg_ms": round(v[0] / v[1], 4), "launches": v[1]} for k, v in timing.items() if v[1]},
    }
    print(json.dumps(out), flush=True)


def bench_trajectory(args):
    """Maintenance over a sequence of adapter updates on the 7B/16K shapes
    (host recovery loop): fresh full recomputation, exact suffix, the drift
    policy and reuse, each on its own copy of the prefix."""
    import torch
    import paper_2609_30884_amd as crf
    import synthetic as syn
    from paper_2609_30884_amd.policy import CalibrationCondition, layer_sensitivity
    from paper_2609_30884_amd.recovery import AdapterVersions, CacheState, Executor, RecoveryLoop, Update
    from synthetic.trajectory import make_calibration_conditions, make_setup, make_state_buffers, new_b
    wl = syn.WORKLOADS["qwen7b_16k"]
    dims, n = wl.dims, wl.window.n_tokens
    t0 = time.perf_counter()
    setup = make_setup(wl, args.seed, n, args.updates)
    cd = crf.make_dims(dims.n_layers, dims.d_model, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.d_ffn,
                       dims.rms_eps, dims.rope_theta, dims.dtype)
    ctx = crf.Context(cd, n, wl.lora_rank)
    weights = crf.layer_weights_array(setup.weights)
    adapters = AdapterVersions(setup.base_lora)
    keep, states = [], {}
    for name in ("fresh", "suffix", "policy"):
        k, v, bnd = make_state_buffers(setup, wl.page_size, args.restart_every)
        keep.append((k, v, bnd))
        states[name] = CacheState(crf.kv_cache(k, v, setup.block_table, n, wl.page_size), bnd,
                                  restart_every=args.restart_every)
    stream = torch.cuda.current_stream()
    ex = Executor(ctx, cd, weights, stream)
    for st in states.values():   # every copy starts as a fresh prefill under version 0
        ex.recompute(st, adapters.array(0), 0, dims.n_layers)
    torch.cuda.synchronize()
    print(f"[bench] trajectory set-up and prefills in {time.perf_counter() - t0:.1f}s", file=sys.stderr, flush=True)
    drift = torch.empty(dims.n_layers, device="cuda")
    risk = torch.empty_like(drift)
    conds = [CalibrationCondition(*c) for c in make_calibration_conditions(wl, args.seed)]
    sens = torch.from_numpy(layer_sensitivity(conds, dims.n_layers).astype("float32")).cuda()
    loop = RecoveryLoop(ex, adapters, dict(states, reuse=None), dims.n_layers, sens, drift, risk)
    g = torch.Generator(device="cuda")
    g.manual_seed(args.seed + 1)
    for i, (layer, target) in enumerate(setup.updates):
        ver = adapters.apply(layer, target, new_b(setup, adapters.versions[-1], layer, target, g))
        recs = loop.step(Update(ver, layer, target))
        pol = next(r for r in recs if r.strategy == "policy")
        print(f"[bench] update {i + 1}/{len(setup.updates)}: {target}@{layer} policy {pol.decision.action} "
              f"[{pol.r},{pol.b}) " + " ".join(f"{r.strategy}={1e3 * r.seconds:.1f}ms" for r in recs),
              file=sys.stderr, flush=True)
    assert ctx.device_errors() == 0
    summ = loop.summary()
    out = {"metric": "maintenance ms over an update trajectory (7B-shape, 16K-token prefix); lower is better",
           "value": summ["policy"]["maintenance_ms"], "unit": "ms", "n_gpus": 1, "steps": len(setup.updates),
           "warmup": 0, "ms_per_step": round(summ["policy"]["maintenance_ms"] / len(setup.updates), 3),
           "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded device draws; one B factor moves by N(0,0.005) per update)",
           "config": {"workload": f"trajectory: {len(setup.updates)} updates, Qwen2.5-7B shapes, {n}-token prefix, "
                                  f"{dims.n_layers} layers, LoRA rank {wl.lora_rank} on {','.join(wl.lora_targets)}, "
                                  f"boundary states retained every {args.restart_every} layer(s)",
                      "updates": [f"{t}@{l}" for l, t in setup.updates]},
           "strategies": summ,
           "sensitivity": [round(float(x), 4) for x in sens.cpu()]}
    print(json.dumps(out), flush=True)


def bench_tail(args):
    """Tail influence at the 7B shapes (Sec. 3.2): the first-step logits z^(b)
    of one new token over a 16K-token prefix whose cache layers before b are
    refreshed under the current adapter and from b on come from an older one,
    for every boundary b = 0..N; the decoding step is timed (HBM-bound)."""
    import numpy as np
    import torch
    import paper_2609_30884_amd as crf
    import synthetic as syn
    from synthetic.trajectory import make_setup, make_state_buffers
    vocab = 152064
    wl = syn.WORKLOADS["qwen7b_16k"]
    dims, n = wl.dims, wl.window.n_tokens
    N = dims.n_layers
    t0 = time.perf_counter()
    setup = make_setup(wl, args.seed, n + 1, 0)
    g = torch.Generator(device="cuda")
    g.manual_seed(args.seed + 2)
    cur = []
    for ll in setup.base_lora:   # the current adapter: every B factor moved by N(0, 0.02)
        tg = {t: (a, (b.float() + 0.02 * torch.randn(b.shape, generator=g, device="cuda")).to(torch.bfloat16))
              for t, (a, b) in ll["targets"].items()}
        cur.append({"rank": ll["rank"], "scale": ll["scale"], "targets": tg})
    fnorm = (1.0 + 0.02 * torch.randn(dims.d_model, generator=g, device="cuda")).to(torch.bfloat16)
    head = (0.02 * torch.randn((vocab, dims.d_model), generator=g, device="cuda")).to(torch.bfloat16)
    x_new = setup.embedding[n:n + 1].contiguous()
    emb = setup.embedding[:n].contiguous()
    cd = crf.make_dims(N, dims.d_model, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.d_ffn,
                       dims.rms_eps, dims.rope_theta, dims.dtype)
    ctx = crf.Context(cd, n + 1, wl.lora_rank)
    weights = crf.layer_weights_array(setup.weights)
    lo_cur, lo_old = crf.lora_array(cur, N), crf.lora_array(setup.base_lora, N)
    pools = {}
    for name, lo in (("fresh", lo_cur), ("stale", lo_old)):
        k, v, _ = make_state_buffers(setup, wl.page_size)
        kv = crf.kv_cache(k, v, setup.block_table, n, wl.page_size)
        crf.recompute_window(ctx, cd, emb, weights, lo, 0, N, kv, None)
        pools[name] = (k, v)
    hk, hv = pools["stale"][0].clone(), pools["stale"][1].clone()
    kvh = crf.kv_cache(hk, hv, setup.block_table, n, wl.page_size)
    logits = torch.empty(vocab, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    print(f"[bench] tail set-up and prefills in {time.perf_counter() - t0:.1f}s", file=sys.stderr, flush=True)
    zs, times = [], []
    for b in range(N + 1):
        if b > 0:   # boundary b: layer b-1 now refreshed
            hk[b - 1].copy_(pools["fresh"][0][b - 1])
            hv[b - 1].copy_(pools["fresh"][1][b - 1])
        for _ in range(max(1, args.warmup) if b == 0 else 0):
            crf.decode_logits(ctx, cd, x_new, weights, lo_cur, kvh, fnorm, head, logits)
        torch.cuda.synchronize()
        reps = max(1, args.steps // 4)
        t1 = time.perf_counter()
        for _ in range(reps):
            crf.decode_logits(ctx, cd, x_new, weights, lo_cur, kvh, fnorm, head, logits)
        torch.cuda.synchronize()
        times.append((time.perf_counter() - t1) / reps)
        zs.append(logits.double().cpu().numpy())
    assert ctx.device_errors() == 0
    z_star = zs[-1]
    v = [np.linalg.norm(zs[l] - zs[l + 1]) for l in range(N)]
    T = [float(sum(v[b:])) for b in range(N + 1)]

    def kl(a, c):
        la = a - (a.max() + np.log(np.exp(a - a.max()).sum()))
        lc = c - (c.max() + np.log(np.exp(c - c.max()).sum()))
        return float(np.sum(np.exp(la) * (la - lc)))
    kls = [kl(z_star, z) for z in zs]
    top1 = [bool(np.argmax(z) == np.argmax(z_star)) for z in zs]
    ms = 1e3 * float(np.median(times))
    w_bytes = N * 2 * (dims.d_model * (dims.dq + 2 * dims.dkv) + dims.dq * dims.d_model + 3 * dims.d_model * dims.d_ffn)
    bytes_step = w_bytes + vocab * dims.d_model * 2 + N * 2 * n * dims.dkv * 2
    out = {"metric": "first-step decode latency over a 16K-token hybrid cache (7B shapes, 152064-token head)",
           "value": round(ms, 3), "unit": "ms", "n_gpus": 1, "steps": N + 1, "warmup": args.warmup,
           "ms_per_step": round(ms, 3), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
           "dtype": "bf16", "data": "synthetic (seeded device draws; current adapter = every B + N(0, 0.02))",
           "config": {"workload": f"tail: one new token over a {n}-token prefix, {N} layers, hybrid boundary b = 0..{N}",
                      "vocab": vocab},
           "roofline": {"bound": "hbm", "kernel": "decode step (all kernels)",
                        "achieved": round(bytes_step / (ms * 1e-3) / 1e9, 1), "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                        "frac": round(bytes_step / (ms * 1e-3) / PEAK_HBM, 4), "traffic": None},
           "tail": {"T_b": [round(x, 4) for x in T], "kl": [float(f"{x:.4g}") for x in kls],
                    "kl_bound_holds": all(k <= 0.25 * t * t + 1e-9 for k, t in zip(kls, T)), "top1_agree": top1}}
    print(json.dumps(out), flush=True)


def bench_copy(args):
    """A plain elementwise pass of known size (1 GiB read, 1 GiB written): the
    calibration point that turns the FETCH_SIZE / WRITE_SIZE counters into
    bytes for the traffic figure of the roofline."""
    import torch
    n = 1 << 28                                    # fp32 elements: 1 GiB
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    elapsed, _ = _timed(lambda: torch.neg(src, out=dst), args.steps, args.warmup)
    bytes_per = 2 * 4 * n
    out = {"metric": "device copy bandwidth (elementwise pass, 1 GiB in + 1 GiB out)",
           "value": round(bytes_per * args.steps / elapsed / 1e9, 1), "unit": "GB/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(1e3 * elapsed / args.steps, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": "copy: 2^28 fp32 elements read and written once per step",
                      "bytes_read": 4 * n, "bytes_written": 4 * n}}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
