"""Thin host-side recovery policy around crf_layer_drift and crf_recompute_window.

The runtime decision of the method (paper Sec. 4.1 "Runtime risk and range
selection"; Sec. 4.2 "Cache and anchor updates"):

* every cached layer l carries the adapter version that produced its K/V
  (its anchor); the cache is a mixed-version object;
* after an update the device computes d_l = ||theta_t - theta_anchor(l)||_2 and
  q_l = s_l d_l (Eq. 8, crf_layer_drift);
* layers with q_l >= 1 trigger; none triggered -> direct reuse; otherwise the
  window end is b_t = 1 + max{l : q_l >= 1} (Eq. 9) and [r, b_t) is
  recomputed from the executable restart r; b_t = N is the exact affected
  suffix, anything shorter is bounded recovery;
* only the recomputed layers' anchors move to the current version.

The earliest cache layer an update can change depends on the module
(supplementary Eq. sup-first-invalid-cache-layer): s for K/V updates,
min(s+1, N) for Q/O/MLP updates (N = no cached layer invalidated); the
executable restart is s whenever a later layer can be affected.

The sensitivities s_l come from offline calibration (Sec. 4.1 "Offline
calibration", Eqs. layer-recovery-label and layer-sensitivity): each
calibration condition i (restart r_i, adapter distance d_i) evaluates the
candidate windows H_i; the first safe one h*_i labels the layers it covers;
per layer, delta_l is the order statistic of the covering conditions'
distances just past a 5% lower tail, and s_l = 1 / delta_l (0 for a layer no
selected window covers).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Iterable, List, Mapping, Optional, Sequence, Tuple

import numpy as np

KV_MODULES = ("k", "v")
QOMLP_MODULES = ("q", "o", "gate", "up", "down", "mlp")


def first_invalid_cache_layer(module: str, s: int, n_layers: int) -> int:
    """r_KV(m, s): s for key/value updates, min(s+1, N) for query/output/MLP updates."""
    if module in KV_MODULES:
        return s
    if module in QOMLP_MODULES:
        return min(s + 1, n_layers)
    raise ValueError(f"unknown update module {module!r}")


def executable_restart(module: str, s: int, n_layers: int) -> Optional[int]:
    """Restart layer for an update of `module` at layer s, or None when no cached
    layer can be affected (the end-boundary sentinel N)."""
    if first_invalid_cache_layer(module, s, n_layers) >= n_layers:
        return None
    return s


@dataclass(frozen=True)
class Decision:
    action: str              # "reuse", "bounded" or "exact_suffix"
    r: int                   # restart layer (inclusive)
    b: int                   # window end (exclusive); b == r for reuse
    triggered: Tuple[int, ...]

    @property
    def h(self) -> int:
        return self.b - self.r

    def fraction(self, n_layers: int) -> float:
        """Normalised recomputation fraction (b - r) / N (Sec. 4.2)."""
        return self.h / n_layers


def decide(risk: Sequence[float], r: Optional[int], n_layers: int) -> Decision:
    """Range selection of Eq. 9 from the per-layer risk q_l.  Ties trigger (q = 1)."""
    q = np.asarray(risk, dtype=np.float64)
    trig = tuple(int(l) for l in np.nonzero(q >= 1.0)[0])
    if r is None or not trig:
        rr = n_layers if r is None else r
        return Decision("reuse", rr, rr, trig)
    b = 1 + max(trig)
    if b <= r:
        return Decision("reuse", r, r, trig)
    return Decision("exact_suffix" if b == n_layers else "bounded", r, b, trig)


@dataclass
class MixedVersionCache:
    """Per-layer anchor versions of one cached prefix (Sec. 4.2)."""
    n_layers: int
    anchor: np.ndarray = field(default=None)

    def __post_init__(self):
        if self.anchor is None:
            self.anchor = np.zeros(self.n_layers, dtype=np.int32)

    def refresh(self, d: Decision, version: int):
        """Anchors move only for the recomputed layers [r, b)."""
        if d.h > 0:
            self.anchor[d.r:d.b] = version

    def stale_layers(self, version: int) -> List[int]:
        return [int(l) for l in np.nonzero(self.anchor != version)[0]]


# ----------------------------------------------------------------------------- offline calibration

CANDIDATE_H = (0, 1, 2, 4, 8, 16)
SAFE_KL, SAFE_TOP1, SAFE_SCORE_DROP = 0.05, 0.99, 0.01
DELTA_TAIL, DELTA_FLOOR = 0.05, 1e-12


def candidate_windows(r: int, n_layers: int) -> List[int]:
    """H_i = {min(h, N - r) : h in {0, 1, 2, 4, 8, 16}} U {N - r}, ascending."""
    rest = n_layers - r
    return sorted({min(h, rest) for h in CANDIDATE_H} | {rest})


def is_safe(kl: float, top1_agreement: float, score_drop: float) -> bool:
    """A candidate is safe against fresh recomputation when first-step
    next-token KL <= 0.05, top-1 agreement >= 0.99 and the full-answer task
    score drops by at most 0.01."""
    return kl <= SAFE_KL and top1_agreement >= SAFE_TOP1 and score_drop <= SAFE_SCORE_DROP


def first_safe_window(safe: Mapping[int, bool]) -> Optional[int]:
    """h* = min{h in H : S(h) = 1} (larger windows need not stay safe); None if none is."""
    ok = [h for h, v in safe.items() if v]
    return min(ok) if ok else None


@dataclass(frozen=True)
class CalibrationCondition:
    r: int                 # restart layer
    d: float               # l2 distance between the active adapter and the stale cache's adapter state
    h_star: Optional[int]  # first safe window (None: no evaluated window was safe)


def recovery_labels(cond: CalibrationCondition, n_layers: int) -> np.ndarray:
    """y_{i,l} = 1[r_i <= l < r_i + h*_i]."""
    y = np.zeros(n_layers, dtype=bool)
    if cond.h_star:
        y[cond.r:cond.r + cond.h_star] = True
    return y


def layer_sensitivity(conditions: Iterable[CalibrationCondition], n_layers: int) -> np.ndarray:
    """s_l = 1 / delta_l with delta_l = max(d_{l,(floor(0.05 n_l) + 1)}, 1e-12), the
    (1-based) order statistic of D_l^+ = {d_i : y_{i,l} = 1}; s_l = 0 when D_l^+ is empty."""
    conds = list(conditions)
    s = np.zeros(n_layers, dtype=np.float64)
    for l in range(n_layers):
        dl = np.sort([c.d for c in conds if recovery_labels(c, n_layers)[l]])
        n = len(dl)
        if n == 0:
            continue
        delta = max(float(dl[int(np.floor(DELTA_TAIL * n))]), DELTA_FLOOR)
        s[l] = 1.0 / delta
    return s
