"""Pins of the oracle's first-step decode, tail influence and the paper's
certificates (Sec. 3.2, Eqs. tail-influence, tail-kl-certificate,
top1-certificate), on tiny random models.  CPU only."""
import dataclasses

import numpy as np
import pytest

import synthetic as syn
from oracle import oracle as O

WL = syn.WORKLOADS["tiny_f32"]
DIMS = WL.dims
VOCAB = 300


def _model(seed, version, wl=WL):
    w = {l: syn.gen_layer_weights(wl, seed, l) for l in range(wl.dims.n_layers)}
    lo = {l: syn.gen_lora_layer(wl, seed, l, version) for l in range(wl.dims.n_layers)}
    g, head = syn.gen_head(wl, seed, VOCAB)
    return w, lo, g, head


def test_rope_at_matches_rope_and_is_relative():
    rng = np.random.default_rng(0)
    x = rng.normal(size=(9, 3, 64))
    assert np.allclose(O.rope_at(x, np.arange(9), 1e6), O.rope(x, 1e6), atol=1e-14)
    q, k = rng.normal(size=(1, 1, 64)), rng.normal(size=(1, 1, 64))
    a = np.sum(O.rope_at(q, np.array([20]), 1e4) * O.rope_at(k, np.array([15]), 1e4))
    b = np.sum(O.rope_at(q, np.array([105]), 1e4) * O.rope_at(k, np.array([100]), 1e4))
    assert a == pytest.approx(b, rel=1e-10)


def test_decode_over_prefill_cache_equals_longer_prefill():
    """Decoding m tokens over the cache of an n-token prefill is the last m rows
    of a prefill over the n + m tokens (definition of KV caching)."""
    seed, n, m = 3, 40, 5
    w, lo, g, head = _model(seed, 1)
    emb = syn.gen_hidden(WL, seed, n + m)
    h_all, kv_all, hs_all = O.prefill(emb, w, lo, DIMS)
    _, kv_pre, _ = O.prefill(emb[:n], w, lo, DIMS)
    h = emb[n:]
    for l in range(DIMS.n_layers):
        h, k, v = O.decode_layer(h, kv_pre[l][0], kv_pre[l][1], w[l], lo[l], DIMS)
        assert np.allclose(k, kv_all[l][0][n:], rtol=1e-10, atol=1e-12)
        assert np.allclose(v, kv_all[l][1][n:], rtol=1e-10, atol=1e-12)
        assert np.allclose(h, hs_all[l][n:], rtol=1e-10, atol=1e-12)
    z = O.decode_logits(emb[n:], kv_pre, w, lo, DIMS, g, head)
    zref = O.rms_norm(h_all[-1:], g, DIMS.rms_eps) @ head.T
    assert np.allclose(z, zref[0], rtol=1e-10, atol=1e-12)


def test_kl_divergence_definition():
    rng = np.random.default_rng(1)
    a, b = rng.normal(size=50) * 3, rng.normal(size=50) * 3
    p, q = np.exp(a) / np.exp(a).sum(), np.exp(b) / np.exp(b).sum()
    assert O.kl_divergence(a, b) == pytest.approx(float(np.sum(p * np.log(p / q))), rel=1e-12)
    assert O.kl_divergence(a, a + 7.0) == pytest.approx(0.0, abs=1e-14)     # shift invariance


def _hybrid_logits(seed, stale_version, n=48, m=3, db=None):
    """z^(b) for b = 0..N: current adapter, fresh caches before b, caches of
    an older adapter from b on."""
    wl = WL if db is None else dataclasses.replace(WL, lora_scale=db)
    w, lo_new, g, head = _model(seed, 3, wl)
    lo_old = {l: syn.gen_lora_layer(wl, seed, l, stale_version) for l in range(DIMS.n_layers)}
    emb = syn.gen_hidden(wl, seed, n)
    x = syn.gen_new_tokens(wl, seed, m)
    _, fresh, _ = O.prefill(emb, w, lo_new, DIMS, wl.lora_scale)
    _, stale, _ = O.prefill(emb, w, lo_old, DIMS, wl.lora_scale)
    N = DIMS.n_layers
    return [O.decode_logits(x, O.hybrid_caches(fresh, stale, b, N), w, lo_new, DIMS, g, head, wl.lora_scale)
            for b in range(N + 1)]


@pytest.mark.parametrize("seed,stale,scale", [(7, 0, 1.0), (17, 1, 30.0), (29, 0, 300.0)])
def test_tail_kl_and_top1_certificates(seed, stale, scale):
    zs = _hybrid_logits(seed, stale, db=scale)
    T = O.tail_influence(zs)
    z_star = zs[-1]
    N = DIMS.n_layers
    assert T[N] == 0.0 and np.all(np.diff(T) <= 1e-15)            # monotone envelope, zero at b = N
    assert np.allclose(zs[0] - z_star, sum(zs[l] - zs[l + 1] for l in range(N)))   # telescoping
    srt = np.sort(z_star)
    margin = srt[-1] - srt[-2]
    for b in range(N + 1):
        kl = O.kl_divergence(z_star, zs[b])
        assert kl <= 0.25 * T[b] ** 2 + 1e-12, (b, kl, T[b])
        if T[b] < margin / 2:
            assert np.argmax(zs[b]) == np.argmax(z_star)
    if scale > 1:
        assert T[0] > 0 and O.kl_divergence(z_star, zs[0]) > 0


def test_fully_fresh_boundary_is_exact():
    zs = _hybrid_logits(7, 3)          # the stale adapter is the current one
    assert all(np.array_equal(z, zs[-1]) for z in zs)
