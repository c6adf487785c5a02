"""Scheduler Engine of the oracle: when to start preparation.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The prefetching-window trade-off model (Section 4.1, Eqs. 3-8) and the
online window selection (Section 4.2, Eq. 9 and Algorithm 1), the
admission check (Section 4.2), smoothing of the telemetry rates (Section
4.2) and the bound on discarded preparation (Section 4.4, Eq. 10), in the
paper's notation, with plain Python floats.

Readings where the paper is silent:
* the candidate set {0, dT, ..., T_limit} is the multiples of dT up to
  T_limit, closed by T_limit itself when T_limit is not a multiple;
* among windows of equal cost the smallest wins (the earliest
  commitment is the latest trigger);
* the smoothing is an exponentially weighted average whose first sample
  sets the value; its weight is a parameter;
* "the request state expected at handover" for admission is the KV cache
  of K_curr + r_d T_remain tokens.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional


@dataclass(frozen=True)
class Rates:
    """Runtime estimates and constants of one migration session."""
    r_p: float          # target prefill throughput available to the session, tokens/s
    r_d: float          # source per-request decode throughput, tokens/s
    B: float            # inter-gNB goodput, bytes/s
    s_kv: float         # KV bytes per token (Eq. 1)
    T_load: float = 0.0  # model load time at the target, s
    T_0: float = 0.0    # activation latency after the state is available, s
    alpha: float = 0.8  # objective weight (the evaluation uses 0.8)
    T_max: float = 5.0  # cap on the window, s
    dT: float = 0.01    # candidate granularity, s


@dataclass
class Window:
    T_w: float
    L_hist: float
    T_hist: float
    S_inc: float
    T_res: float
    T_SIT: float
    T_early: float
    J: float


def evaluate(rt: Rates, K_curr: float, T_remain: float, T_w: float) -> Window:
    """Eqs. 9, 4, 3, 5, 6, 7, 8 at one candidate window."""
    L_hist = K_curr + rt.r_d * (T_remain - T_w)            # Eq. 9: prefix at the candidate trigger
    T_hist = rt.T_load + L_hist / rt.r_p                   # Eq. 4
    S_inc = rt.r_d * T_w * rt.s_kv                         # Eq. 3
    T_res = max(0.0, S_inc / rt.B - T_w)                   # Eq. 5
    T_SIT = rt.T_0 + max(0.0, T_hist - T_w, T_res)         # Eq. 6
    T_early = max(0.0, T_w - T_hist)                       # Eq. 7
    J = rt.alpha * T_SIT + (1.0 - rt.alpha) * T_early      # Eq. 8
    return Window(T_w, L_hist, T_hist, S_inc, T_res, T_SIT, T_early, J)


def candidates(T_limit: float, dT: float) -> List[float]:
    """The set W = {0, dT, ..., T_limit} of Algorithm 1."""
    W = [min(k * dT, T_limit) for k in range(int(math.floor(T_limit / dT)) + 1)]
    if T_limit - W[-1] > 1e-12 * max(1.0, T_limit):
        W.append(T_limit)
    return W


@dataclass
class Decision:
    best: Window
    n_candidates: int
    trigger: bool


def select(rt: Rates, K_curr: float, T_remain: float) -> Decision:
    """Algorithm 1 after the admission check: T_limit = min(T_max,
    T_remain), evaluate J over W, keep the argmin, trigger when T_remain
    <= T_w*, otherwise defer to the next control cycle."""
    T_limit = min(rt.T_max, max(T_remain, 0.0))
    W = candidates(T_limit, rt.dT)
    best: Optional[Window] = None
    for T_w in W:
        w = evaluate(rt, K_curr, T_remain, T_w)
        if best is None or w.J < best.J:
            best = w
    return Decision(best, len(W), T_remain <= best.T_w)


def ewma(prev: Optional[float], sample: float, weight: float) -> float:
    """Smoothed estimate after one sample (None: no sample yet)."""
    return sample if prev is None else weight * sample + (1.0 - weight) * prev


def admit(compatible: bool, vram_free: float, s_kv: float, K_curr: float, r_d: float,
          T_remain: float) -> bool:
    """The target runs a compatible model and holds the request state
    expected at handover."""
    return bool(compatible) and vram_free >= s_kv * (K_curr + r_d * max(T_remain, 0.0))


def waste_bound(T_max: float, E_early: float, T_avail: float) -> float:
    """Eq. 10."""
    return max(T_max + E_early - T_avail, 0.0)
