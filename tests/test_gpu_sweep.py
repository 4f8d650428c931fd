"""A seeded sweep of small bf16 model shapes against the oracle: head sizes,
GQA group sizes, widths, d_ffn multiples of 64, adapter ranks 8..64 on random
target subsets, prefix lengths from 1 to 1800 and window placements.  The
configurations are drawn once from a fixed seed, so every run checks the same
ones."""
import dataclasses

import numpy as np
import pytest

import synthetic as syn
from tests.helpers import assert_window_parity, oracle_window, run_gpu_window

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _configs(n=12, seed=2609):
    rng = np.random.Generator(np.random.PCG64(seed))
    out = []
    while len(out) < n:
        hd = int(rng.choice([64, 128]))
        n_kv = int(rng.choice([2, 4]) if hd == 64 else rng.choice([1, 2, 4]))
        group = int(rng.choice([1, 2, 3, 4, 6, 7]))
        n_q = n_kv * group
        if (n_q * hd) % 128:
            continue
        d_model = int(rng.choice([256, 384, 512, 768, 1024]))
        d_ffn = 64 * int(rng.integers(5, 41))
        rank = int(rng.choice([8, 16, 24, 32, 48, 64]))
        k = int(rng.integers(1, len(syn.TARGETS) + 1))
        targets = tuple(sorted(rng.choice(syn.TARGETS, size=k, replace=False), key=syn.TARGETS.index))
        n_tok = int(rng.choice([int(rng.integers(1, 40)), int(rng.integers(40, 600)), int(rng.integers(600, 1800))]))
        l0 = int(rng.integers(0, 2))
        h = int(rng.integers(1, 4 - l0 + 1))
        out.append(dict(head_dim=hd, n_kv_heads=n_kv, n_q_heads=n_q, d_model=d_model, d_ffn=d_ffn, rank=rank,
                        targets=targets, n=n_tok, l0=l0, h=h))
    return out


CONFIGS = _configs()


def _id(c):
    return (f"hd{c['head_dim']}-q{c['n_q_heads']}kv{c['n_kv_heads']}-d{c['d_model']}-f{c['d_ffn']}-r{c['rank']}"
            f"-{'+'.join(c['targets'])}-n{c['n']}-l{c['l0']}h{c['h']}")


@pytest.mark.parametrize("cfg", CONFIGS, ids=[_id(c) for c in CONFIGS])
def test_bf16_shape_sweep(cfg):
    from synthetic.device import build_case
    base = syn.WORKLOADS["qwen7b_16k"].with_dims(n_layers=4, d_model=cfg["d_model"], n_q_heads=cfg["n_q_heads"],
                                                  n_kv_heads=cfg["n_kv_heads"], head_dim=cfg["head_dim"],
                                                  d_ffn=cfg["d_ffn"])
    wl = dataclasses.replace(base.with_window(n_tokens=cfg["n"], l0=cfg["l0"], h=cfg["h"]), lora_rank=cfg["rank"],
                             lora_targets=cfg["targets"])
    print(f"[case] sweep {_id(cfg)}", flush=True)
    case = build_case(wl, 43)
    run_gpu_window(case)
    torch.cuda.synchronize()
    out, kv = oracle_window(case)
    assert_window_parity(case, out, kv, label=_id(cfg))


def _f32_configs(n=4, seed=884):
    rng = np.random.Generator(np.random.PCG64(seed))
    out = []
    for _ in range(n):
        hd = int(rng.choice([64, 128]))
        n_kv = int(rng.choice([1, 2]))
        n_q = n_kv * int(rng.choice([1, 2, 3]))
        out.append(dict(head_dim=hd, n_kv_heads=n_kv, n_q_heads=n_q, d_model=8 * int(rng.integers(8, 49)),
                        d_ffn=8 * int(rng.integers(8, 120)), rank=int(rng.choice([0, 4, 8, 12])),
                        n=int(rng.integers(1, 300)), l0=int(rng.integers(0, 2)), h=int(rng.integers(1, 3))))
    return out


F32_CONFIGS = _f32_configs()


@pytest.mark.parametrize("cfg", F32_CONFIGS, ids=[
    f"hd{c['head_dim']}-q{c['n_q_heads']}kv{c['n_kv_heads']}-d{c['d_model']}-f{c['d_ffn']}-r{c['rank']}-n{c['n']}"
    f"-l{c['l0']}h{c['h']}" for c in F32_CONFIGS])
def test_f32_shape_sweep(cfg):
    """The fp32 path on widths and d_ffn that are only multiples of 8, ranks
    0-12 on every target."""
    from synthetic.device import build_case
    base = syn.WORKLOADS["tiny_f32"].with_dims(n_layers=4, d_model=cfg["d_model"], n_q_heads=cfg["n_q_heads"],
                                                n_kv_heads=cfg["n_kv_heads"], head_dim=cfg["head_dim"],
                                                d_ffn=cfg["d_ffn"])
    wl = dataclasses.replace(base.with_window(n_tokens=cfg["n"], l0=cfg["l0"], h=cfg["h"]), lora_rank=cfg["rank"],
                             lora_targets=syn.TARGETS if cfg["rank"] else ())
    print(f"[case] f32 sweep {cfg}", flush=True)
    case = build_case(wl, 47)
    run_gpu_window(case)
    torch.cuda.synchronize()
    out, kv = oracle_window(case)
    assert_window_parity(case, out, kv, label=f"f32 {cfg}")


def _decode_configs(n=4, seed=3088):
    rng = np.random.Generator(np.random.PCG64(seed))
    out = []
    while len(out) < n:
        hd = int(rng.choice([64, 128]))
        n_kv = int(rng.choice([2, 4]) if hd == 64 else rng.choice([1, 2, 4]))
        n_q = n_kv * int(rng.choice([1, 2, 4, 6, 7]))
        if (n_q * hd) % 128:
            continue
        shape = dict(n_layers=2, d_model=int(rng.choice([256, 512, 768, 1024])), n_q_heads=n_q, n_kv_heads=n_kv,
                     head_dim=hd, d_ffn=64 * int(rng.integers(5, 41)))
        out.append((shape, int(rng.integers(1, 2500)), int(rng.integers(1, 17))))
    return out


DECODE_CONFIGS = _decode_configs()


@pytest.mark.parametrize("shape,n,m", DECODE_CONFIGS, ids=[
    f"hd{s['head_dim']}-q{s['n_q_heads']}kv{s['n_kv_heads']}-d{s['d_model']}-f{s['d_ffn']}-n{n}-m{m}"
    for s, n, m in DECODE_CONFIGS])
def test_decode_shape_sweep(shape, n, m):
    """First decoding step (m new tokens over an n-token cache, hybrid at
    boundary 1) on random shapes, through the skinny projections and the
    key-split attention."""
    from tests.test_gpu_decode import _check_decode
    _check_decode(19, n, m, 1, base="qwen7b_16k", shape=shape, vocab=1024)
