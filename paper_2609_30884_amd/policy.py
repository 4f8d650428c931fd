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
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

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
