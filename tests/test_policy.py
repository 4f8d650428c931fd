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


# ----------------------------------------------------------------------------- offline calibration (Sec. 4.1)

from paper_2609_30884_amd.policy import (CalibrationCondition, candidate_windows, first_safe_window, is_safe,
                                          layer_sensitivity, recovery_labels)


def test_candidate_windows():
    assert candidate_windows(0, 28) == [0, 1, 2, 4, 8, 16, 28]
    assert candidate_windows(20, 28) == [0, 1, 2, 4, 8]        # min(16, 8) = 8 = N - r
    assert candidate_windows(27, 28) == [0, 1]
    assert candidate_windows(10, 28) == [0, 1, 2, 4, 8, 16, 18]


def test_safety_thresholds_and_first_safe_window():
    assert is_safe(0.05, 0.99, 0.01) and not is_safe(0.0501, 1.0, 0.0)
    assert not is_safe(0.0, 0.9899, 0.0) and not is_safe(0.0, 1.0, 0.0101)
    # larger windows need not remain safe: the first safe one is taken
    assert first_safe_window({0: False, 1: False, 2: True, 4: False, 8: True}) == 2
    assert first_safe_window({0: True, 1: True}) == 0
    assert first_safe_window({0: False, 1: False}) is None


def test_recovery_labels():
    y = recovery_labels(CalibrationCondition(r=3, d=0.5, h_star=2), 8)
    assert list(y) == [False, False, False, True, True, False, False, False]
    assert not recovery_labels(CalibrationCondition(r=3, d=0.5, h_star=0), 8).any()     # direct reuse
    assert not recovery_labels(CalibrationCondition(r=3, d=0.5, h_star=None), 8).any()


def test_sensitivity_order_statistic_by_hand():
    n_layers = 4
    # layer 1 covered by 20 conditions with d = 1..20: floor(0.05 * 20) + 1 = 2nd smallest = 2
    conds = [CalibrationCondition(1, float(d), 1) for d in range(1, 21)]
    # layer 2 covered by 19 conditions: floor(0.95) + 1 = 1st smallest = 3
    conds += [CalibrationCondition(2, float(d), 1) for d in range(3, 22)]
    # layer 3 covered once with d = 0: the floor 1e-12 applies
    conds += [CalibrationCondition(3, 0.0, 1)]
    s = layer_sensitivity(conds, n_layers)
    assert s[0] == 0.0                                       # no selected window covers layer 0
    assert s[1] == pytest.approx(1 / 2.0)
    assert s[2] == pytest.approx(1 / 3.0)
    assert s[3] == pytest.approx(1e12)


def test_sensitivity_forty_conditions_and_window_spans():
    # 40 conditions restarting at 0 with window 2 cover layers 0 and 1: 3rd smallest d
    rng = np.random.default_rng(3)
    d = rng.uniform(0.1, 5.0, 40)
    conds = [CalibrationCondition(0, float(x), 2) for x in d]
    s = layer_sensitivity(conds, 5)
    third = np.sort(d)[2]
    assert s[0] == pytest.approx(1 / third) and s[1] == pytest.approx(1 / third)
    assert (s[2:] == 0).all()


def test_calibrated_sensitivity_drives_the_trigger():
    # small-drift conditions that still needed recovery make a layer sensitive
    conds = [CalibrationCondition(2, 0.1, 2), CalibrationCondition(5, 10.0, 1)]
    s = layer_sensitivity(conds, N)
    assert s[2] == pytest.approx(10.0) and s[5] == pytest.approx(0.1)
    d = np.full(N, 0.2)                     # the same drift everywhere
    q = s * d
    assert q[2] >= 1 and q[3] >= 1 and q[5] < 1
    dec = decide(q, 2, N)
    assert (dec.action, dec.r, dec.b) == ("bounded", 2, 4)
