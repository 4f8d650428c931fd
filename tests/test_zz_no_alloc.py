"""crf_layer_drift_noalloc (the drift call for callers that cannot allocate)
against crf_layer_drift through the C ABI: two calls in a row, the second with
a smaller request, each bitwise equal to the context call on the same inputs
(same kernels in the same order)."""
import numpy as np
import pytest

import synthetic as syn
from tests.helpers import cdims

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

SMALL = dict(n_layers=4, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=64, d_ffn=1024)


def _request(wl, seed, n_versions, keep):
    from synthetic.device import lora_to_dev
    dims = wl.dims
    states = [[syn.gen_lora_layer(wl, seed, l, v) for l in range(dims.n_layers)] for v in range(n_versions + 1)]
    import paper_2609_30884_amd as crf

    def arr(state):
        dev = [lora_to_dev(state[l], wl.lora_rank, 1.0, dims) for l in range(dims.n_layers)]
        keep.append(dev)
        return crf.lora_array(dev, dims.n_layers)

    vers = [arr(s) for s in states[:n_versions]]
    cur = arr(states[n_versions])
    anchors = syn.gen_anchor_versions(dims.n_layers, n_versions, seed)
    sens = torch.from_numpy(syn.gen_sensitivity(dims.n_layers, seed)).cuda()
    return cur, vers, anchors, sens


def _outputs(n_layers, n_versions):
    return (torch.full((n_layers,), float("nan"), device="cuda"), torch.full((n_layers,), float("nan"), device="cuda"),
            torch.full((n_versions * n_layers,), float("nan"), device="cuda"))


@pytest.mark.parametrize("per_layer_only", [0, 1])
def test_drift_noalloc_matches_context_call(per_layer_only):
    import paper_2609_30884_amd as crf
    keep = []
    big = syn.WORKLOADS["qwen15b_mixed8"]
    small = syn.WORKLOADS["qwen7b_16k"].with_dims(**SMALL)
    for wl, n_versions, seed in ((big, 4, 7), (small, 2, 17)):
        dims = wl.dims
        print(f"[case] drift noalloc {wl.name} layers={dims.n_layers} versions={n_versions} "
              f"per_layer_only={per_layer_only}", flush=True)
        cur, vers, anchors, sens = _request(wl, seed, n_versions, keep)
        cd = cdims(dims)
        ctx = crf.Context(cd, 1, wl.lora_rank)
        ref = _outputs(dims.n_layers, n_versions)
        crf.layer_drift(ctx, cd, cur, vers, anchors, sens, *ref, per_layer_only=bool(per_layer_only))
        got = _outputs(dims.n_layers, n_versions)
        crf.layer_drift_noalloc(cd, cur, vers, anchors, sens, *got, per_layer_only=bool(per_layer_only))
        torch.cuda.synchronize()
        for a, b in zip(ref, got):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), (a, b)
        assert bool(torch.isfinite(got[0]).all()) and float(got[0].min()) > 0
        ctx.close()
