"""Host recovery loop over a sequence of adapter updates (paper Sec. 4.1-4.2).

Each update moves one LoRA factor of one layer to a new adapter version.  A
maintained prefix is a mixed-version object: every cached layer carries the
version that produced its K/V (its anchor), and the retained boundary states
H_{l-1} let any layer be a restart point.  Per update and strategy:

* fresh    recompute every layer from the embedding state H_{-1};
* suffix   recompute [r, N) from the executable restart r;
* policy   run crf_layer_drift against the anchors, trigger q_l >= 1 and
           recompute [r, b_t) with b_t = 1 + max{q_l >= 1} (Eq. 9), or reuse;
* reuse    keep the cache (no maintenance).

Only recomputed layers move their anchors to the current version.

Restart boundaries (Sec. 4.2: a restart at r needs the retained state H_{r-1})
are kept every `restart_every` layers (boundaries[l] for l a multiple of it;
1 = every layer).  A restart is rounded down to the nearest retained boundary
(the layers in between see unchanged inputs and weights, so their refreshed
K/V equal the cached ones), and a window runs as one crf_recompute_window call
per span between retained boundaries: the span's output goes to the next
retained boundary, and a span that ends at the window end off a boundary runs
without an output state (its last layer needs only its K/V projections).  The
compute is crf_recompute_window / crf_layer_drift.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from . import _lib as L
from .policy import Decision, decide, executable_restart

STRATEGIES = ("fresh", "suffix", "policy", "reuse")


@dataclass(frozen=True)
class Update:
    """One adapter update: the factor B of `target` at `layer` moves (the new version is `version`)."""
    version: int
    layer: int
    target: str


class AdapterVersions:
    """Every version of an adapter whose updates each replace one factor.

    versions[v][l] is the per-layer dict {"rank", "scale", "targets": {name: (A, B)}}
    of device tensors; versions share the tensors an update did not replace."""

    def __init__(self, base: Sequence[Optional[dict]]):
        self.versions: List[List[Optional[dict]]] = [list(base)]
        self._arrays: Dict[int, object] = {}

    @property
    def current(self) -> int:
        return len(self.versions) - 1

    def apply(self, layer: int, target: str, new_b) -> int:
        prev = self.versions[-1]
        nxt = list(prev)
        ll = dict(prev[layer])
        tg = dict(ll["targets"])
        a, _ = tg[target]
        tg[target] = (a, new_b)
        ll["targets"] = tg
        nxt[layer] = ll
        self.versions.append(nxt)
        return self.current

    def array(self, v: int):
        if v not in self._arrays:
            self._arrays[v] = L.lora_array(self.versions[v], len(self.versions[v]))
        return self._arrays[v]


@dataclass
class CacheState:
    """One maintained prefix: paged K/V of every layer (kv), the retained
    boundary states (boundaries[l] = H_{l-1}, boundaries[0] = H_{-1}; None
    where l is not a multiple of restart_every), the per-layer anchor
    versions and the spacing of the retained boundaries."""
    kv: object
    boundaries: list
    anchor: np.ndarray = field(default=None)
    restart_every: int = 1

    def __post_init__(self):
        if self.anchor is None:
            self.anchor = np.zeros(len(self.boundaries) - 1, dtype=np.int32)
        if self.restart_every < 1:
            raise ValueError("restart_every must be >= 1")

    def restart(self, r: Optional[int]) -> Optional[int]:
        """The retained boundary a restart at layer r starts from."""
        return None if r is None else r - r % self.restart_every

    def spans(self, r: int, b: int):
        """(start, end, output boundary index or None) of the calls covering [r, b)."""
        k = self.restart_every
        if r % k:
            raise ValueError(f"restart {r} is not a retained boundary (every {k} layers)")
        out, l = [], r
        while l < b:
            e = min(l + k, b)
            out.append((l, e, e if (e % k == 0 or e == len(self.boundaries) - 1) else None))
            l = e
        return out


@dataclass
class StepRecord:
    strategy: str
    update: Update
    r: Optional[int]
    b: Optional[int]
    layers: int
    seconds: float
    decision: Optional[Decision] = None


class Executor:
    """The GPU calls a strategy makes (kept separate so the loop logic can be
    exercised on the host with a stand-in)."""

    def __init__(self, ctx, dims, weights, stream=None):
        self.ctx, self.dims, self.weights, self.stream = ctx, dims, weights, stream

    def recompute(self, state: CacheState, lora_array, r: int, b: int):
        for l0, e, out in state.spans(r, b):
            L.recompute_window(self.ctx, self.dims, state.boundaries[l0], self.weights, lora_array, l0, e - l0,
                               state.kv, None if out is None else state.boundaries[out], self.stream)

    def risk(self, adapters: AdapterVersions, anchor: np.ndarray, sensitivity, drift_out, risk_out) -> np.ndarray:
        used = sorted(set(int(a) for a in anchor))
        index = {v: i for i, v in enumerate(used)}
        L.layer_drift(self.ctx, self.dims, adapters.array(adapters.current), [adapters.array(v) for v in used],
                      [index[int(a)] for a in anchor], sensitivity, drift_out, risk_out, stream=self.stream)
        return risk_out.float().cpu().numpy().astype(np.float64)

    def synchronize(self):
        import torch
        torch.cuda.synchronize()


class RecoveryLoop:
    """Drives the four strategies over a shared sequence of updates."""

    def __init__(self, executor: Executor, adapters: AdapterVersions, states: Dict[str, Optional[CacheState]],
                 n_layers: int, sensitivity, drift_out=None, risk_out=None):
        self.ex, self.adapters, self.states, self.n = executor, adapters, states, n_layers
        self.sensitivity, self.drift_out, self.risk_out = sensitivity, drift_out, risk_out
        self.records: List[StepRecord] = []

    def _timed(self, fn: Callable[[], None]) -> float:
        self.ex.synchronize()
        t0 = time.perf_counter()
        fn()
        self.ex.synchronize()
        return time.perf_counter() - t0

    def step(self, upd: Update) -> List[StepRecord]:
        n, v = self.n, upd.version
        arr = self.adapters.array(v)
        out = []
        r_exec = executable_restart(upd.target, upd.layer, n)
        for name, st in self.states.items():
            r = st.restart(r_exec) if st is not None else r_exec
            if name == "fresh":
                dt = self._timed(lambda: self.ex.recompute(st, arr, 0, n))
                st.anchor[:] = v
                out.append(StepRecord(name, upd, 0, n, n, dt))
            elif name == "suffix":
                if r is None:
                    out.append(StepRecord(name, upd, None, None, 0, 0.0))
                    continue
                dt = self._timed(lambda: self.ex.recompute(st, arr, r, n))
                st.anchor[r:] = v
                out.append(StepRecord(name, upd, r, n, n - r, dt))
            elif name == "policy":
                box = {}

                def run():
                    if r is None:
                        box["d"] = Decision("reuse", n, n, ())
                        return
                    q = self.ex.risk(self.adapters, st.anchor, self.sensitivity, self.drift_out, self.risk_out)
                    d = decide(q, r, n)
                    box["d"] = d
                    if d.h > 0:
                        self.ex.recompute(st, arr, d.r, d.b)

                dt = self._timed(run)
                d = box["d"]
                if d.h > 0:
                    st.anchor[d.r:d.b] = v
                out.append(StepRecord(name, upd, d.r, d.b, d.h, dt, d))
            elif name == "reuse":  # the state may be None: nothing is maintained
                out.append(StepRecord(name, upd, None, None, 0, 0.0))
            else:
                raise ValueError(f"unknown strategy {name!r}")
        self.records.extend(out)
        return out

    def summary(self) -> Dict[str, dict]:
        res = {}
        for name in self.states:
            rs = [x for x in self.records if x.strategy == name]
            n_upd = max(len(rs), 1)
            res[name] = {
                "maintenance_ms": round(1e3 * sum(x.seconds for x in rs), 3),
                "layers_recomputed": int(sum(x.layers for x in rs)),
                "fraction": round(sum(x.layers for x in rs) / (n_upd * self.n), 4),
            }
            if name == "policy":
                res[name]["actions"] = {a: sum(1 for x in rs if x.decision and x.decision.action == a)
                                        for a in ("reuse", "bounded", "exact_suffix")}
        return res
