"""Host checks of the ideal-bf16 error model (tests/golden/bf16_model.py) that
the bf16 parity bounds rest on."""
import json
import math

import numpy as np
import pytest

import synthetic as syn
from tests.golden import bf16_model as M
from tests.helpers import MODEL_HEADROOM, MODEL_RUNS, TOL, TOL_ELEM, stored_model_elem_max

SMALL = dict(n_layers=4, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=64, d_ffn=1024)


def _small(h=2, n=200, targets=syn.TARGETS):
    import dataclasses
    wl = syn.WORKLOADS["qwen7b_16k"].with_dims(**SMALL).with_window(n_tokens=n, l0=1, h=h)
    return dataclasses.replace(wl, lora_targets=targets)


def test_model_without_rounding_is_the_oracle():
    """With its bf16 rounding switched off the model is the oracle's window in
    fp32 arithmetic: every tensor agrees to fp32 accuracy."""
    e = M.window_errors(_small(h=3), rnd=M._ident)
    assert max(a for a, _ in e.values()) < 2e-6
    assert max(b for _, b in e.values()) < 2e-5


def test_rounding_one_tensor_costs_at_most_half_an_ulp():
    """Closed form: rounding to bf16 (8-bit significand) moves an element by at
    most half an ulp, at most 2^-8 of its magnitude, i.e. at most
    2^-8 max|T| / rms(T) in the element metric; on a Gaussian-like tensor of
    10^7 elements that alone is 1-2e-2."""
    rng = np.random.default_rng(3)
    t = rng.standard_normal(10 ** 7).astype(np.float32)
    _, elem = M.errors(M._bf16(t), t)
    bound = 2.0 ** -8 * float(np.max(np.abs(t))) / math.sqrt(float(np.mean(t.astype(np.float64) ** 2)))
    assert elem <= bound * (1 + 1e-6)
    assert 1e-2 < elem < 2.5e-2


def test_model_errors_are_bf16_sized():
    """The rounded model sits a bf16 step away from the oracle: far above fp32
    noise, within the relative RMS bound for a three-layer window."""
    e = M.window_errors(_small(h=3))
    rms = max(a for a, _ in e.values())
    assert 5e-4 < rms < TOL["bf16"] / MODEL_HEADROOM
    assert max(b for _, b in e.values()) < TOL_ELEM["bf16"]


def test_stored_runs_and_derived_bounds():
    """The stored full-size runs cover the windows the bounds are taken from;
    ideal execution stays below 2e-2 relative RMS for windows of up to three
    layers; the element bound used without a model run is the headroom times
    the largest stored element error."""
    runs = json.load(open(MODEL_RUNS))
    for name in ("qwen15b_4k", "qwen7b_16k"):
        r = runs[name]
        w = syn.WORKLOADS[name].window
        assert (r["n_tokens"], r["l0"], r["h"], r["seed"]) == (w.n_tokens, w.l0, w.h, M.SEED)
        keys = {f"{t}{l}" for l in range(w.l0, w.l0 + w.h) for t in "KV"} | {"hidden_out"}
        assert set(r["errors"]) == keys
        assert max(e["rms_rel"] for e in r["errors"].values()) < TOL["bf16"]
    assert TOL_ELEM["bf16"] == pytest.approx(MODEL_HEADROOM * stored_model_elem_max())
    assert 2e-2 < stored_model_elem_max() < 4e-2


def test_stored_run_reproduces():
    """Recomputing the stored 1.5B-shaped 4K window gives the stored figures."""
    stored = json.load(open(MODEL_RUNS))["qwen15b_4k"]["errors"]
    e = M.window_errors(syn.WORKLOADS["qwen15b_4k"])
    for k, (a, b) in e.items():
        assert a == pytest.approx(stored[k]["rms_rel"], rel=2e-2)
        assert b == pytest.approx(stored[k]["elem"], rel=5e-2)


def test_model_rms_match_notices_planted_deviations():
    """The GPU tests require the GPU's relative RMS error to equal the model's to
    within MODEL_RMS_MATCH.  Planted in the model, an extra bf16 rounding of the
    residual stream after each update, or a missing rounding of the normalised
    inputs or of the stored K or V (the dominant terms), moves that ratio past
    it on some tensor; the other rounding points (U, Q, P, the attention and
    SwiGLU outputs) weigh too little in these errors for the check to see them."""
    from tests.helpers import MODEL_RMS_MATCH
    wl = _small(h=2)
    base = M.window_errors(wl)
    for variant in ("resid_bf16", "skip_x", "skip_k", "skip_v"):
        e = M.window_errors(wl, variant=variant)
        worst = max(abs(e[k][0] / base[k][0] - 1.0) for k in base)
        assert worst > 3 * MODEL_RMS_MATCH, (variant, worst)
    for variant in M.VARIANTS:  # every planted deviation keeps the window bf16-sized
        e = M.window_errors(wl, variant=variant)
        assert max(a for a, _ in e.values()) < TOL["bf16"]
