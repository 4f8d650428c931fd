"""Host recovery loop on the GPU (Sec. 4.1-4.2): fresh, exact-suffix and
policy maintenance of three copies of one prefix over a sequence of adapter
updates.  The exact suffix from the executable restart must leave the cache
bitwise equal to fresh recomputation after every update (layers before the
restart are unaffected by the update, and the same kernels see the same
inputs); the policy's anchors move only inside its windows."""
import dataclasses

import numpy as np
import pytest

import synthetic as syn
from tests.helpers import bits_equal, cdims

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.mark.parametrize("restart_every", [1, 2])
def test_recovery_trajectory_small(restart_every):
    import paper_2609_30884_amd as crf
    from paper_2609_30884_amd.policy import CalibrationCondition, layer_sensitivity
    from paper_2609_30884_amd.recovery import AdapterVersions, CacheState, Executor, RecoveryLoop, Update
    from synthetic.trajectory import make_calibration_conditions, make_setup, make_state_buffers, new_b
    wl = dataclasses.replace(syn.WORKLOADS["qwen15b_4k"], lora_targets=syn.TARGETS).with_dims(
        n_layers=6, d_model=256, n_q_heads=2, n_kv_heads=1, head_dim=128, d_ffn=512)
    n, n_upd = 200, 8
    setup = make_setup(wl, 7, n, n_upd)
    N = wl.dims.n_layers
    print(f"[case] recovery trajectory N={N} n={n} updates={setup.updates} restart_every={restart_every}",
          flush=True)
    cd = cdims(wl.dims)
    ctx = crf.Context(cd, n, wl.lora_rank)
    weights = crf.layer_weights_array(setup.weights)
    adapters = AdapterVersions(setup.base_lora)
    bufs, states = {}, {}
    for name in ("fresh", "suffix", "policy"):
        k, v, bnd = make_state_buffers(setup, wl.page_size, restart_every)
        bufs[name] = (k, v)
        states[name] = CacheState(crf.kv_cache(k, v, setup.block_table, n, wl.page_size), bnd,
                                  restart_every=restart_every)
    ex = Executor(ctx, cd, weights)
    for st in states.values():
        ex.recompute(st, adapters.array(0), 0, N)
    torch.cuda.synchronize()
    assert bits_equal(bufs["suffix"][0], bufs["fresh"][0])
    drift = torch.empty(N, device="cuda")
    risk = torch.empty(N, device="cuda")
    conds = [CalibrationCondition(*c) for c in make_calibration_conditions(wl, 7)]
    sens = torch.from_numpy(layer_sensitivity(conds, N).astype(np.float32)).cuda()
    loop = RecoveryLoop(ex, adapters, dict(states, reuse=None), N, sens, drift, risk)
    g = torch.Generator(device="cuda")
    g.manual_seed(123)
    for layer, target in setup.updates:
        ver = adapters.apply(layer, target, new_b(setup, adapters.versions[-1], layer, target, g))
        pol_before = states["policy"].anchor.copy()
        recs = {r.strategy: r for r in loop.step(Update(ver, layer, target))}
        torch.cuda.synchronize()
        assert bits_equal(bufs["suffix"][0], bufs["fresh"][0]) and bits_equal(bufs["suffix"][1], bufs["fresh"][1])
        d = recs["policy"].decision
        moved = np.nonzero(states["policy"].anchor != pol_before)[0]
        if d.h > 0:
            assert set(moved) <= set(range(d.r, d.b)) and (states["policy"].anchor[d.r:d.b] == ver).all()
        else:
            assert len(moved) == 0
        assert np.isfinite(risk.cpu().numpy()).all() or d.action == "reuse"
    assert ctx.device_errors() == 0
    summ = loop.summary()
    print(f"[recovery] {summ}", flush=True)
    assert summ["fresh"]["fraction"] == 1.0
    assert summ["suffix"]["layers_recomputed"] <= summ["fresh"]["layers_recomputed"]


def _host(t):
    return t.float().cpu().numpy()


def test_recovery_policy_matches_oracle_trajectory():
    """The policy strategy over 8 updates, side by side with the same loop on
    the CPU oracle (Eq. 8 risk from oracle.layer_drift, the same host
    decision, Eq. 9 window end, each window's layers from oracle.decoder_layer
    starting at the retained boundary, Sec. 4.2 anchor updates): equal risks,
    trigger sets and window ends at every update, and the final mixed-version
    cache equal to the oracle's layer by layer."""
    import paper_2609_30884_amd as crf
    from oracle import oracle as O
    from paper_2609_30884_amd.policy import CalibrationCondition, decide, executable_restart, layer_sensitivity
    from paper_2609_30884_amd.recovery import AdapterVersions, CacheState, Executor, RecoveryLoop, Update
    from synthetic.device import gather_kv
    from synthetic.trajectory import make_calibration_conditions, make_setup, make_state_buffers, new_b
    from tests.helpers import TOL, TOL_ELEM, rel_to_rms, rms_rel
    wl = dataclasses.replace(syn.WORKLOADS["qwen15b_4k"], lora_targets=syn.TARGETS).with_dims(
        n_layers=6, d_model=256, n_q_heads=2, n_kv_heads=1, head_dim=128, d_ffn=512)
    n, n_upd = 200, 8
    setup = make_setup(wl, 29, n, n_upd)
    dims, N = wl.dims, wl.dims.n_layers
    print(f"[case] recovery vs oracle N={N} n={n} updates={setup.updates}", flush=True)
    cd = cdims(dims)
    ctx = crf.Context(cd, n, wl.lora_rank)
    weights = crf.layer_weights_array(setup.weights)
    adapters = AdapterVersions(setup.base_lora)
    k, v, bnd = make_state_buffers(setup, wl.page_size)
    st = CacheState(crf.kv_cache(k, v, setup.block_table, n, wl.page_size), bnd)
    ex = Executor(ctx, cd, weights)
    ex.recompute(st, adapters.array(0), 0, N)
    drift = torch.empty(N, device="cuda")
    risk = torch.full((N,), float("nan"), device="cuda")
    conds = [CalibrationCondition(*c) for c in make_calibration_conditions(wl, 7)]
    sens_np = layer_sensitivity(conds, N).astype(np.float32)
    loop = RecoveryLoop(ex, adapters, {"policy": st}, N, torch.from_numpy(sens_np).cuda(), drift, risk)

    # the oracle's copy of the same prefix: host weights and adapter versions
    # (the values the GPU holds), fp64 cache, boundaries and anchors
    W = [{key: _host(t) for key, t in w.items()} for w in setup.weights]
    host_versions = [[{t: (_host(a), _host(b)) for t, (a, b) in ll["targets"].items()} for ll in setup.base_lora]]
    emb = _host(setup.embedding)
    _, kv_ref, hs = O.prefill(emb, W, dict(enumerate(host_versions[0])), dims, wl.lora_scale)
    bnd_ref = [emb.astype(np.float64)] + [hs[l] for l in range(N)]
    anchor_ref = np.zeros(N, dtype=np.int32)
    g = torch.Generator(device="cuda")
    g.manual_seed(321)
    bt = setup.block_table.cpu().numpy()
    actions = []
    for layer, target in setup.updates:
        b_new = new_b(setup, adapters.versions[-1], layer, target, g)
        ver = adapters.apply(layer, target, b_new)
        cur = [dict(x) for x in host_versions[-1]]
        cur[layer] = dict(cur[layer])
        cur[layer][target] = (cur[layer][target][0], _host(b_new))
        host_versions.append(cur)
        risk.fill_(float("nan"))
        rec = {r_.strategy: r_ for r_ in loop.step(Update(ver, layer, target))}["policy"]
        torch.cuda.synchronize()
        # the oracle's decision from its own anchors (the GPU passes only the versions in use)
        r = executable_restart(target, layer, N)
        if r is None:
            d_ref = decide(np.zeros(N), None, N)
        else:
            used = sorted(set(int(a) for a in anchor_ref))
            idx = {u: i for i, u in enumerate(used)}
            _, q_ref, _ = O.layer_drift(cur, [host_versions[u] for u in used], [idx[int(a)] for a in anchor_ref],
                                        sens_np.astype(np.float64))
            q_gpu = _host(risk).astype(np.float64)
            assert np.allclose(q_gpu, q_ref, rtol=2e-6, atol=0), (q_gpu, q_ref)
            d_ref = decide(q_ref, r, N)
            near = np.abs(q_ref - 1.0) < 1e-6
            if not near.any():
                assert rec.decision.triggered == d_ref.triggered
        assert (rec.decision.r, rec.decision.b, rec.decision.action) == (d_ref.r, d_ref.b, d_ref.action)
        actions.append(d_ref.action)
        for l in range(d_ref.r, d_ref.b):
            h_l, k_l, v_l = O.decoder_layer(bnd_ref[l], W[l], cur[l], dims, wl.lora_scale)
            bnd_ref[l + 1] = h_l
            kv_ref[l] = (k_l, v_l)
        anchor_ref[d_ref.r:d_ref.b] = ver
        assert np.array_equal(st.anchor, anchor_ref)
    print(f"[recovery] actions {actions} anchors {anchor_ref.tolist()}", flush=True)
    assert "bounded" in actions or "exact_suffix" in actions
    errs = {}
    for l in range(N):
        for nm, pool, ref in (("K", k, kv_ref[l][0]), ("V", v, kv_ref[l][1])):
            got = gather_kv(pool, l, bt, n, wl.page_size)
            errs[f"{nm}{l}"] = (rms_rel(got, ref), rel_to_rms(got, ref))
    print("[parity] recovery cache " + " ".join(f"{key}=({a:.2e},{b:.2e})" for key, (a, b) in errs.items()),
          flush=True)
    bad = {key: e for key, e in errs.items() if not (e[0] <= TOL["bf16"] and e[1] <= TOL_ELEM["bf16"])}
    assert not bad, bad
    assert ctx.device_errors() == 0
