"""Pins for the oracle: closed forms, invariants, brute force and independent
library implementations.  CPU only.

Each pin is chosen so that a plausible slip in the oracle (a dropped term, a
wrong sign, a wrong head map, a transposed operand) fails at least one test;
`test_mutations_are_caught` plants such slips in the oracle and checks that.
"""
import math

import numpy as np
import pytest
import torch

import synthetic as syn
from oracle import brute
from oracle import oracle as O

RNG = np.random.default_rng(1234)


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.sqrt(np.mean(b * b)), 1e-300))


# ---------------------------------------------------------------------------- RMSNorm

def test_rmsnorm_matches_torch_and_invariants():
    x = RNG.standard_normal((7, 48))
    g = 1 + 0.1 * RNG.standard_normal(48)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (48,), torch.tensor(g), eps=1e-6).numpy()
    assert rel(O.rms_norm(x, g, 1e-6), ref) < 1e-14
    # unit-RMS rows for g = 1, eps = 0; scale invariance for c > 0
    y = O.rms_norm(x, np.ones(48), 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=1)), 1.0, atol=1e-14)
    assert rel(O.rms_norm(3.7 * x, g, 0.0), O.rms_norm(x, g, 0.0)) < 1e-14
    # eps sits inside the root: a zero row stays zero, a tiny row is damped
    z = O.rms_norm(np.full((1, 4), 1e-4), np.ones(4), 1e-6)
    assert np.allclose(z, 1e-4 / math.sqrt(1e-8 + 1e-6))


# ---------------------------------------------------------------------------- RoPE

def test_rope_closed_form_complex_rotation():
    n, heads, hd, theta = 9, 3, 16, 1e6
    x = RNG.standard_normal((n, heads, hd))
    got = O.rope(x, theta)
    z = x[..., :hd // 2] + 1j * x[..., hd // 2:]
    inv = theta ** (-np.arange(0, hd, 2) / hd)
    phi = np.arange(n)[:, None] * inv[None, :]
    zr = z * np.exp(1j * phi)[:, None, :]
    exp = np.concatenate([zr.real, zr.imag], axis=-1)
    assert rel(got, exp) < 1e-14


def test_rope_invariants():
    n, hd = 33, 64
    x = RNG.standard_normal((n, 2, hd))
    y = O.rope(x, 1e6)
    assert np.array_equal(y[0], x[0])                          # position 0 is the identity
    pn = lambda t: t[..., :hd // 2] ** 2 + t[..., hd // 2:] ** 2
    assert np.allclose(pn(y), pn(x), rtol=1e-13)               # pair norms preserved
    # <R_p q, R_s k> depends only on p - s
    q = RNG.standard_normal(hd)
    k = RNG.standard_normal(hd)
    qs = O.rope(np.tile(q, (n, 1, 1)), 1e4)[:, 0]
    ks = O.rope(np.tile(k, (n, 1, 1)), 1e4)[:, 0]
    assert abs(qs[20] @ ks[13] - qs[9] @ ks[2]) < 1e-11
    assert abs(qs[20] @ ks[13] - qs[7] @ ks[0]) < 1e-11
    # brute-force per-element rotation
    for p in (0, 5, 32):
        assert np.allclose(brute.rope_vec(list(x[p, 1]), p, 1e6), y[p, 1], atol=1e-13)


def test_rope_matches_transformers_qwen2():
    from transformers import Qwen2Config
    from transformers.models.qwen2.modeling_qwen2 import Qwen2RotaryEmbedding, apply_rotary_pos_emb
    cfg = Qwen2Config(hidden_size=128, num_attention_heads=2, num_key_value_heads=1, rope_theta=1e6,
                      max_position_embeddings=4096)
    cfg.rope_parameters = {"rope_type": "default", "rope_theta": 1e6}
    emb = Qwen2RotaryEmbedding(cfg)
    n = 300
    x = RNG.standard_normal((n, 2, 64))
    pos = torch.arange(n)[None]
    cos, sin = emb(torch.zeros(1, n, 64, dtype=torch.float64), pos)
    qt = torch.tensor(x).transpose(0, 1)[None]  # [1, heads, n, hd]
    qr, _ = apply_rotary_pos_emb(qt, qt, cos.double(), sin.double())
    ref = qr[0].transpose(0, 1).numpy()
    # transformers builds its angles in fp32; allow that rounding
    assert rel(O.rope(x, 1e6), ref) < 5e-5


# ---------------------------------------------------------------------------- LoRA

def test_lora_linear_identities():
    x = RNG.standard_normal((5, 24))
    w = RNG.standard_normal((10, 24))
    a = RNG.standard_normal((4, 24))
    b = RNG.standard_normal((10, 4))
    merged = w + 0.5 * (b @ a)                       # x (W + s B A)^T
    assert rel(O.lora_linear(x, w, (a, b), 0.5), x @ merged.T) < 1e-13
    assert np.array_equal(O.lora_linear(x, w, (a, np.zeros_like(b))), O.lora_linear(x, w))
    bias = RNG.standard_normal(10)
    assert rel(O.lora_linear(x, w, None, 1.0, bias), x @ w.T + bias) < 1e-14


# ---------------------------------------------------------------------------- attention

def _sdpa(q, k, v):
    qt = torch.tensor(q).permute(1, 0, 2)[None]
    kt = torch.tensor(k).permute(1, 0, 2)[None]
    vt = torch.tensor(v).permute(1, 0, 2)[None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True, enable_gqa=True)
    return o[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("nq,nkv", [(4, 2), (6, 1), (3, 3), (7, 1)])
def test_attention_matches_sdpa_and_brute(nq, nkv):
    n, hd = 13, 8
    q, k, v = (RNG.standard_normal((n, h, hd)) for h in (nq, nkv, nkv))
    got = O.causal_gqa_attention(q, k, v, q_block=5)
    assert rel(got, _sdpa(q, k, v)) < 1e-13
    bo = brute.attention(q.tolist(), k.tolist(), v.tolist(), nq, nkv, hd)
    assert rel(got, np.array(bo)) < 1e-13


def test_attention_closed_forms():
    n, nq, nkv, hd = 40, 4, 2, 16
    q, k, v = (RNG.standard_normal((n, h, hd)) for h in (nq, nkv, nkv))
    o = O.causal_gqa_attention(q, k, v, q_block=7)
    for j in range(nq):                                  # row 0 sees only key 0
        assert np.allclose(o[0, j], v[0, j // 2], atol=1e-15)
    o0 = O.causal_gqa_attention(np.zeros_like(q), k, v)  # Q = 0: causal running mean
    run = np.cumsum(v, axis=0) / np.arange(1, n + 1)[:, None, None]
    for j in range(nq):
        assert np.allclose(o0[:, j], run[:, j // 2], atol=1e-13)
    # GQA = MHA on repeated K/V (head j uses group j // (nq/nkv))
    kr, vr = np.repeat(k, 2, axis=1), np.repeat(v, 2, axis=1)
    assert rel(O.causal_gqa_attention(q, kr, vr), o) < 1e-14
    # query blocking changes nothing
    assert rel(O.causal_gqa_attention(q, k, v, q_block=1000), o) < 1e-14


def test_silu():
    x = RNG.standard_normal(100) * 4
    assert rel(O.silu(x), torch.nn.functional.silu(torch.tensor(x)).numpy()) < 1e-14


# ---------------------------------------------------------------------------- whole layer

def _tiny_dims(**kw):
    base = dict(n_layers=4, d_model=64, n_q_heads=4, n_kv_heads=2, head_dim=16, d_ffn=96, dtype="f32")
    base.update(kw)
    return syn.Dims(**base)


def _rand_layer(dims, rng, bias=False, rank=4, targets=syn.TARGETS):
    w = {"attn_norm": 1 + 0.1 * rng.standard_normal(dims.d_model),
         "mlp_norm": 1 + 0.1 * rng.standard_normal(dims.d_model)}
    for t in syn.TARGETS:
        w["w_" + t] = 0.1 * rng.standard_normal(dims.target_shape(t))
    if bias:
        for t in ("q", "k", "v"):
            w["bias_" + t] = 0.3 * rng.standard_normal(dims.target_shape(t)[0])
    lora = {}
    for t in targets:
        d_out, d_in = dims.target_shape(t)
        lora[t] = (0.3 * rng.standard_normal((rank, d_in)), 0.1 * rng.standard_normal((d_out, rank)))
    return w, lora


def _hf_layer(dims, w, lora, scale):
    from transformers import Qwen2Config
    from transformers.models.qwen2.modeling_qwen2 import Qwen2DecoderLayer
    cfg = Qwen2Config(hidden_size=dims.d_model, intermediate_size=dims.d_ffn, num_attention_heads=dims.n_q_heads,
                      num_key_value_heads=dims.n_kv_heads, head_dim=dims.head_dim, rms_norm_eps=dims.rms_eps,
                      num_hidden_layers=1, max_position_embeddings=4096)
    cfg.rope_parameters = {"rope_type": "default", "rope_theta": dims.rope_theta}
    cfg._attn_implementation = "eager"
    layer = Qwen2DecoderLayer(cfg, 0).double()
    names = {"q": layer.self_attn.q_proj, "k": layer.self_attn.k_proj, "v": layer.self_attn.v_proj,
             "o": layer.self_attn.o_proj, "gate": layer.mlp.gate_proj, "up": layer.mlp.up_proj,
             "down": layer.mlp.down_proj}
    with torch.no_grad():
        for t, mod in names.items():
            m = w["w_" + t].copy()
            if t in lora:
                a, b = lora[t]
                m = m + scale * (b @ a)                  # merged weight W + s B A
            mod.weight.copy_(torch.tensor(m))
            if mod.bias is not None:
                bb = w.get("bias_" + t)
                mod.bias.copy_(torch.tensor(bb if bb is not None else np.zeros(mod.weight.shape[0])))
        layer.input_layernorm.weight.copy_(torch.tensor(w["attn_norm"]))
        layer.post_attention_layernorm.weight.copy_(torch.tensor(w["mlp_norm"]))
    return cfg, layer


def _hf_run(dims, w, lora, scale, h):
    from transformers.cache_utils import DynamicCache
    from transformers.models.qwen2.modeling_qwen2 import Qwen2RotaryEmbedding
    cfg, layer = _hf_layer(dims, w, lora, scale)
    n = h.shape[0]
    emb = Qwen2RotaryEmbedding(cfg)
    pos = torch.arange(n)[None]
    cos, sin = emb(torch.zeros(1, n, dims.head_dim, dtype=torch.float64), pos)
    mask = torch.full((n, n), float("-inf"), dtype=torch.float64).triu(1)[None, None]
    cache = DynamicCache(config=cfg)
    with torch.no_grad():
        out = layer(torch.tensor(h)[None], attention_mask=mask, position_ids=pos, past_key_values=cache,
                    use_cache=True, position_embeddings=(cos.double(), sin.double()))
    out = out[0] if isinstance(out, tuple) else out
    kk = cache.layers[0].keys[0].permute(1, 0, 2).numpy()
    vv = cache.layers[0].values[0].permute(1, 0, 2).numpy()
    return out[0].numpy(), kk, vv


@pytest.mark.parametrize("bias,scale", [(False, 1.0), (True, 0.5)])
def test_decoder_layer_matches_transformers_qwen2(bias, scale):
    dims = _tiny_dims()
    rng = np.random.default_rng(77)
    w, lora = _rand_layer(dims, rng, bias=bias)
    h = rng.standard_normal((37, dims.d_model))
    ho, k, v = O.decoder_layer(h, w, lora, dims, scale)
    rh, rk, rv = _hf_run(dims, w, lora, scale, h)
    # transformers' RMSNorm and RoPE tables run in fp32 internally
    assert rel(ho, rh) < 2e-6
    assert rel(k, rk) < 2e-6
    assert rel(v, rv) < 2e-6


def test_decoder_layer_matches_brute():
    dims = _tiny_dims(d_model=16, head_dim=4, d_ffn=24, n_q_heads=4, n_kv_heads=2)
    rng = np.random.default_rng(5)
    w, lora = _rand_layer(dims, rng, bias=True, rank=2)
    h = rng.standard_normal((6, dims.d_model))
    ho, k, v = O.decoder_layer(h, w, lora, dims, 0.7)
    bh, bk, bv = brute.decoder_layer(h.tolist(), w, lora, dims, 0.7)
    assert rel(ho, np.array(bh)) < 1e-12
    assert rel(k, np.array(bk)) < 1e-12
    assert rel(v, np.array(bv)) < 1e-12


# ---------------------------------------------------------------------------- window invariants

def _model(dims, seed, n_layers=None, perturb_from=None, perturb_targets=syn.TARGETS):
    """weights, old LoRA and new LoRA (new = old + N(0, 0.05) on B of perturbed layers)."""
    rng = np.random.default_rng(seed)
    W, L_old, L_new = {}, {}, {}
    for l in range(dims.n_layers):
        w, lora = _rand_layer(dims, rng)
        W[l], L_old[l] = w, lora
        if perturb_from is None or l >= perturb_from:
            L_new[l] = {t: (a, b + (0.05 * rng.standard_normal(b.shape) if t in perturb_targets else 0.0))
                        for t, (a, b) in lora.items()}
        else:
            L_new[l] = lora
    return W, L_old, L_new


def test_zero_delta_reproduces_stale_cache():
    """Recomputing with the adapter that produced the cache reproduces it
    (Sec. 4.2: ordinary decoder execution, no correction)."""
    dims = _tiny_dims()
    W, L_old, _ = _model(dims, 1)
    emb = np.random.default_rng(2).standard_normal((29, dims.d_model))
    Hn, KV, Hs = O.prefill(emb, W, L_old, dims)
    out, kv = O.recompute_window(Hs[0], W, L_old, 1, 2, dims)
    for l in (1, 2):
        assert np.array_equal(kv[l][0], KV[l][0]) and np.array_equal(kv[l][1], KV[l][1])
    assert np.array_equal(out, Hs[2])
    # B = 0 on both sides is the same statement for a zero adapter delta
    Z = {l: syn.zero_lora_like(L_old[l]) for l in L_old}
    _, KVz, Hz = O.prefill(emb, W, Z, dims)
    outz, kvz = O.recompute_window(Hz[1], W, Z, 2, 2, dims)
    assert np.array_equal(kvz[3][0], KVz[3][0]) and np.array_equal(outz, Hz[3])


def test_exact_suffix_equals_fresh_prefill():
    """With the update confined to layers >= l0, recomputing [l0, N) from the
    retained boundary equals fresh prefill under the new adapter, and the
    layers before l0 are unchanged (Sec. 2.2; supplementary Sec. S1.1)."""
    dims = _tiny_dims()
    l0 = 2
    W, L_old, L_new = _model(dims, 3, perturb_from=l0)
    emb = np.random.default_rng(4).standard_normal((31, dims.d_model))
    _, KV_old, H_old = O.prefill(emb, W, L_old, dims)
    Hn_new, KV_new, _ = O.prefill(emb, W, L_new, dims)
    out, kv = O.recompute_window(H_old[l0 - 1], W, L_new, l0, dims.n_layers - l0, dims)
    for l in range(dims.n_layers):
        if l < l0:
            assert np.array_equal(KV_old[l][0], KV_new[l][0])
        else:
            assert np.array_equal(kv[l][0], KV_new[l][0]) and np.array_equal(kv[l][1], KV_new[l][1])
            assert not np.array_equal(kv[l][0], KV_old[l][0])
    assert np.array_equal(out, Hn_new)


@pytest.mark.parametrize("targets", [("q",), ("o",), ("gate", "up", "down")])
def test_q_o_mlp_update_leaves_same_layer_kv(targets):
    """A query, output or MLP update at layer s does not change layer s's K/V
    (supplementary Eq. sup-first-invalid-cache-layer: r_KV = s+1 for Q/O/MLP)."""
    dims = _tiny_dims()
    s = 1
    W, L_old, L_new = _model(dims, 6, perturb_from=s, perturb_targets=targets)
    emb = np.random.default_rng(8).standard_normal((17, dims.d_model))
    _, KV_old, H_old = O.prefill(emb, W, L_old, dims)
    out, kv = O.recompute_window(H_old[s - 1], W, L_new, s, 1, dims)
    assert np.array_equal(kv[s][0], KV_old[s][0]) and np.array_equal(kv[s][1], KV_old[s][1])
    assert not np.allclose(out, H_old[s])
    # ... while a K or V update at s does change it (r_KV = s)
    W, L_old, L_new = _model(dims, 6, perturb_from=s, perturb_targets=("v",))
    _, KV_old, H_old = O.prefill(emb, W, L_old, dims)
    _, kv = O.recompute_window(H_old[s - 1], W, L_new, s, 1, dims)
    assert not np.array_equal(kv[s][1], KV_old[s][1])


def test_causal_prefix_invariance_and_composition():
    dims = _tiny_dims()
    W, _, L = _model(dims, 9)
    h = np.random.default_rng(10).standard_normal((50, dims.d_model))
    full, kvf = O.recompute_window(h, W, L, 1, 3, dims)
    part, kvp = O.recompute_window(h[:23], W, L, 1, 3, dims)
    assert rel(part, full[:23]) < 1e-12
    for l in (1, 2, 3):
        assert rel(kvp[l][0], kvf[l][0][:23]) < 1e-12
    a, kva = O.recompute_window(h, W, L, 1, 1, dims)
    b, kvb = O.recompute_window(a, W, L, 2, 2, dims)
    assert np.array_equal(b, full)
    assert np.array_equal(kvb[3][1], kvf[3][1]) and np.array_equal(kva[1][0], kvf[1][0])
    # h = 0 is direct reuse
    z, kvz = O.recompute_window(h, W, L, 2, 0, dims)
    assert np.array_equal(z, h) and kvz == {}


# ---------------------------------------------------------------------------- drift

def _adapters(n_layers, rng, shapes):
    return [{t: (rng.standard_normal(sa), rng.standard_normal(sb)) for t, (sa, sb) in shapes.items()}
            for _ in range(n_layers)]


def test_drift_closed_form_and_invariants():
    rng = np.random.default_rng(11)
    shapes = {"q": ((2, 3), (4, 2)), "v": ((2, 3), (2, 2))}
    cur = _adapters(3, rng, shapes)
    v0 = _adapters(3, rng, shapes)
    d, q, sq = O.layer_drift(cur, [v0, cur], [0, 1, 0], sensitivity=[2.0, 5.0, 0.5])
    # closed form: whole-adapter l2 distance to the anchor version
    flat = lambda ad: np.concatenate([np.concatenate([a.ravel(), b.ravel()]) for layer in ad
                                      for t, (a, b) in sorted(layer.items())])
    dist = np.linalg.norm(flat(cur) - flat(v0))
    assert np.allclose(d, [dist, 0.0, dist], rtol=1e-14)
    assert np.allclose(q, [2 * dist, 0.0, 0.5 * dist], rtol=1e-14)
    assert np.allclose(sq[0].sum(), dist ** 2, rtol=1e-14) and np.all(sq[1] == 0)
    # per-layer slice reading
    dl, _, _ = O.layer_drift(cur, [v0], [0, 0, 0], per_layer_only=True)
    for l in range(3):
        sl = np.concatenate([np.concatenate([(cur[l][t][0] - v0[l][t][0]).ravel(),
                                             (cur[l][t][1] - v0[l][t][1]).ravel()]) for t in sorted(shapes)])
        assert np.isclose(dl[l], np.linalg.norm(sl), rtol=1e-14)
    # +delta then -delta returns to the anchor: drift cancels
    delta = [{t: (0 * a, rng.standard_normal(b.shape)) for t, (a, b) in layer.items()} for layer in cur]
    plus = [{t: (a + delta[l][t][0], b + delta[l][t][1]) for t, (a, b) in cur[l].items()} for l in range(3)]
    back = [{t: (a - delta[l][t][0], b - delta[l][t][1]) for t, (a, b) in plus[l].items()} for l in range(3)]
    dz, _, _ = O.layer_drift(back, [cur], [0, 0, 0])
    assert np.all(dz < 1e-12)


# ---------------------------------------------------------------------------- mutations

def test_mutations_are_caught(monkeypatch):
    """Plant plausible mistakes in the oracle (CPU only) and check that the
    independent transformers pin rejects each one."""
    dims = _tiny_dims()
    rng = np.random.default_rng(21)
    w, lora = _rand_layer(dims, rng)
    h = rng.standard_normal((19, dims.d_model))
    rh, rk, rv = _hf_run(dims, w, lora, 1.0, h)

    def off(**patches):
        with monkeypatch.context() as m:
            for name, fn in patches.items():
                m.setattr(O, name, fn)
            ho, k, v = O.decoder_layer(h, w, lora, dims, 1.0)
        return max(rel(ho, rh), rel(k, rk), rel(v, rv))

    orig_rope, orig_attn, orig_norm, orig_lin = O.rope, O.causal_gqa_attention, O.rms_norm, O.lora_linear

    def _rope_bad(x, theta):  # sign error in the second half
        y = orig_rope(x, theta)
        hd = x.shape[-1]
        c, s = O.rope_angles(x.shape[0], hd, theta)
        x1, x2 = x[..., :hd // 2], x[..., hd // 2:]
        return np.concatenate([y[..., :hd // 2], x2 * c[:, None] - x1 * s[:, None]], axis=-1)

    def attn_bad_map(q, k, v, q_block=1024):  # head j -> group j % nkv
        nq, nkv = q.shape[1], k.shape[1]
        perm = [j % nkv for j in range(nq)]
        return orig_attn(q, k[:, perm], v[:, perm], q_block)

    def norm_no_eps(x, g, eps):
        return orig_norm(x, g, 0.0) * 1.0001

    def lin_no_lora(x, w_, lora_=None, scale=1.0, bias=None):
        return orig_lin(x, w_, None, scale, bias)

    def lin_delta_sign(x, w_, lora_=None, scale=1.0, bias=None):
        return orig_lin(x, w_, lora_, -scale, bias)

    assert off() < 2e-6
    assert off(rope=_rope_bad) > 1e-3
    assert off(causal_gqa_attention=attn_bad_map) > 1e-3
    assert off(rms_norm=norm_no_eps) > 5e-5
    assert off(lora_linear=lin_no_lora) > 1e-3
    assert off(lora_linear=lin_delta_sign) > 1e-3
