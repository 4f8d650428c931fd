"""Host recovery loop (Sec. 4.1-4.2) with a stand-in executor: which windows
each strategy recomputes and how anchors move.  CPU only."""
import numpy as np
import pytest

from paper_2609_30884_amd.recovery import CacheState, RecoveryLoop, Update

N = 8


class FakeExecutor:
    """Risk q_l = s_l * (current version - anchor_l); records recompute calls."""

    def __init__(self, s):
        self.s = np.asarray(s, dtype=np.float64)
        self.calls = []

    def recompute(self, state, lora_array, r, b):
        self.calls.append((id(state), r, b))

    def risk(self, adapters, anchor, sensitivity, drift_out, risk_out):
        return self.s * (adapters.current - anchor.astype(np.float64))

    def synchronize(self):
        pass


class FakeAdapters:
    def __init__(self):
        self.current = 0

    def array(self, v):
        return None


def _loop(s):
    ex = FakeExecutor(s)
    states = {k: CacheState(kv=None, boundaries=[None] * (N + 1)) for k in ("fresh", "suffix", "policy")}
    states["reuse"] = None
    ad = FakeAdapters()
    return ex, ad, states, RecoveryLoop(ex, ad, states, N, sensitivity=None)


def test_strategies_windows_and_anchors():
    s = np.full(N, 0.0)
    s[5] = 0.6      # layer 5 triggers once two versions stale
    ex, ad, states, loop = _loop(s)
    ad.current = 1
    recs = {r.strategy: r for r in loop.step(Update(1, 3, "k"))}
    assert (recs["fresh"].r, recs["fresh"].b, recs["fresh"].layers) == (0, N, N)
    assert (recs["suffix"].r, recs["suffix"].b) == (3, N)
    assert recs["policy"].decision.action == "reuse"        # q_5 = 0.6 < 1
    assert recs["reuse"].layers == 0
    assert list(states["suffix"].anchor) == [0, 0, 0, 1, 1, 1, 1, 1]
    assert list(states["policy"].anchor) == [0] * N
    ad.current = 2
    recs = {r.strategy: r for r in loop.step(Update(2, 2, "q"))}
    d = recs["policy"].decision
    assert (d.action, d.r, d.b) == ("bounded", 2, 6)         # q_5 = 1.2 triggers: b = 6
    assert list(states["policy"].anchor) == [0, 0, 2, 2, 2, 2, 0, 0]
    assert list(states["fresh"].anchor) == [2] * N


def test_final_layer_query_update_needs_no_recompute():
    ex, ad, states, loop = _loop(np.full(N, 10.0))
    ad.current = 1
    recs = {r.strategy: r for r in loop.step(Update(1, N - 1, "o"))}
    assert recs["suffix"].layers == 0 and recs["policy"].layers == 0
    assert recs["policy"].decision.action == "reuse"
    assert recs["fresh"].layers == N
    summ = loop.summary()
    assert summ["fresh"]["fraction"] == 1.0 and summ["suffix"]["layers_recomputed"] == 0
    assert summ["policy"]["actions"]["reuse"] == 1


def test_unknown_strategy_rejected():
    ex = FakeExecutor(np.zeros(N))
    loop = RecoveryLoop(ex, FakeAdapters(), {"bogus": None}, N, sensitivity=None)
    with pytest.raises(ValueError):
        loop.step(Update(1, 0, "q"))


def test_retained_boundaries_spans_and_restarts():
    """With a retained state every k layers, a restart rounds down to a
    retained boundary and a window runs as one call per span between them; a
    span ending at the window end off a boundary writes no output state."""
    st = CacheState(kv=None, boundaries=[None] * (N + 1), restart_every=3)
    assert [st.restart(r) for r in range(N)] == [0, 0, 0, 3, 3, 3, 6, 6]
    assert st.restart(None) is None
    assert st.spans(0, N) == [(0, 3, 3), (3, 6, 6), (6, 8, 8)]      # layer N's output is retained
    assert st.spans(3, 5) == [(3, 5, None)]
    assert st.spans(3, 7) == [(3, 6, 6), (6, 7, None)]
    with pytest.raises(ValueError):
        st.spans(4, 6)
    one = CacheState(kv=None, boundaries=[None] * (N + 1))
    assert one.spans(2, 5) == [(2, 3, 3), (3, 4, 4), (4, 5, 5)]
    with pytest.raises(ValueError):
        CacheState(kv=None, boundaries=[None] * (N + 1), restart_every=0)


def test_policy_restarts_from_retained_boundary():
    s = np.zeros(N)
    s[6] = 2.0
    ex = FakeExecutor(s)
    st = CacheState(kv=None, boundaries=[None] * (N + 1), restart_every=4)
    ad = FakeAdapters()
    loop = RecoveryLoop(ex, ad, {"policy": st, "suffix": CacheState(kv=None, boundaries=[None] * (N + 1),
                                                                     restart_every=4)}, N, sensitivity=None)
    ad.current = 1
    recs = {r.strategy: r for r in loop.step(Update(1, 5, "v"))}
    d = recs["policy"].decision
    assert (d.action, d.r, d.b) == ("bounded", 4, 7)     # restart 5 rounds down to the boundary at 4
    assert (recs["suffix"].r, recs["suffix"].b) == (4, N)
    assert list(st.anchor) == [0, 0, 0, 0, 1, 1, 1, 0]
