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


def test_recovery_trajectory_small():
    import paper_2609_30884_amd as crf
    from paper_2609_30884_amd.policy import CalibrationCondition, layer_sensitivity
    from paper_2609_30884_amd.recovery import AdapterVersions, CacheState, Executor, RecoveryLoop, Update
    from synthetic.trajectory import make_calibration_conditions, make_setup, make_state_buffers, new_b
    wl = dataclasses.replace(syn.WORKLOADS["qwen15b_4k"], lora_targets=syn.TARGETS).with_dims(
        n_layers=6, d_model=256, n_q_heads=2, n_kv_heads=1, head_dim=128, d_ffn=512)
    n, n_upd = 200, 8
    setup = make_setup(wl, 7, n, n_upd)
    N = wl.dims.n_layers
    print(f"[case] recovery trajectory N={N} n={n} updates={setup.updates}", flush=True)
    cd = cdims(wl.dims)
    ctx = crf.Context(cd, n, wl.lora_rank)
    weights = crf.layer_weights_array(setup.weights)
    adapters = AdapterVersions(setup.base_lora)
    bufs, states = {}, {}
    for name in ("fresh", "suffix", "policy"):
        k, v, bnd = make_state_buffers(setup, wl.page_size)
        bufs[name] = (k, v)
        states[name] = CacheState(crf.kv_cache(k, v, setup.block_table, n, wl.page_size), bnd)
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
