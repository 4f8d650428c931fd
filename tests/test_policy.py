"""Host policy: restart layer, trigger, window end and anchor bookkeeping
(Sec. 4.1-4.2; supplementary Eq. sup-first-invalid-cache-layer).  CPU only."""
import numpy as np
import pytest

from paper_2609_30884_amd.policy import (Decision, MixedVersionCache, decide, executable_restart,
                                          first_invalid_cache_layer)

N = 28


@pytest.mark.parametrize("m,s,expect", [("k", 5, 5), ("v", 14, 14), ("q", 5, 6), ("o", 5, 6), ("mlp", 5, 6),
                                        ("gate", 27, 28), ("v", 27, 27), ("down", 0, 1)])
def test_first_invalid_cache_layer(m, s, expect):
    assert first_invalid_cache_layer(m, s, N) == expect


def test_executable_restart_and_sentinel():
    assert executable_restart("q", 10, N) == 10          # restart at s although r_KV = s+1
    assert executable_restart("o", N - 1, N) is None     # final-layer Q/O/MLP update: nothing cached changes
    assert executable_restart("v", N - 1, N) == N - 1
    with pytest.raises(ValueError):
        first_invalid_cache_layer("bias", 1, N)


def test_decide_window_end_and_actions():
    q = np.zeros(N)
    assert decide(q, 14, N).action == "reuse"            # nothing triggered
    q[15] = 0.999999
    assert decide(q, 14, N).action == "reuse"
    q[15] = 1.0                                           # tie triggers
    d = decide(q, 14, N)
    assert (d.action, d.r, d.b, d.h) == ("bounded", 14, 16, 2)
    assert d.fraction(N) == pytest.approx(2 / 28)         # the fixed 2-layer window is 7.14 % of 28 layers
    q[27] = 3.0
    d = decide(q, 14, N)
    assert (d.action, d.b) == ("exact_suffix", N)
    assert d.fraction(N) == pytest.approx(14 / 28)        # 50 % of layers for a middle-layer suffix
    # a trigger below the restart alone does not open a window
    q2 = np.zeros(N)
    q2[3] = 5.0
    assert decide(q2, 14, N).action == "reuse"
    # no restart (sentinel) means reuse whatever the risk
    assert decide(q, None, N).action == "reuse"


def test_anchor_update_only_inside_window():
    c = MixedVersionCache(N)
    c.refresh(Decision("bounded", 14, 16, (15,)), version=3)
    assert list(c.anchor[14:16]) == [3, 3]
    assert c.anchor[:14].sum() == 0 and c.anchor[16:].sum() == 0
    assert c.stale_layers(3) == [l for l in range(N) if l not in (14, 15)]
    c.refresh(Decision("reuse", 14, 14, ()), version=4)
    assert list(c.anchor[14:16]) == [3, 3]
