"""Pins of the oracle's Scheduler Engine (Sections 4.1, 4.2, 4.4) against
closed forms derived from the model, not against its own formulas.

With rho = r_d / r_p the prefix-reconstruction deficit is linear in the
window: T_hist(T_w) - T_w = (1 + rho)(T_c - T_w) with
T_c = (T_load + (K_curr + r_d T_remain) / r_p) / (1 + rho), the window at
which reconstruction finishes exactly at handover.  With beta =
r_d s_kv / B the backlog is T_res = max(0, (beta - 1) T_w).  So:
* with no backlog (beta <= 1), J = alpha (T_0 + (1 + rho)(T_c - T_w))
  below T_c and alpha T_0 + (1 - alpha)(1 + rho)(T_w - T_c) above it: the
  best candidate is one of the two grid points around T_c;
* with alpha = 1 every window from T_c on costs T_0, so the first grid point
  at or after T_c wins;
* with alpha = 0 the zero window costs nothing;
* with a backlog (beta > 1) and alpha = 1, T_SIT - T_0 is the larger of two
  lines that cross at T_x = (1 + rho) T_c / (beta + rho)."""
import math

import numpy as np
import pytest

from oracle import scheduler as sch

RNG = np.random.default_rng(2608)


def random_rates(alpha, backlog=False, dT=0.05):
    r_p = float(RNG.uniform(500, 20000))
    r_d = float(RNG.uniform(5, 80))
    s_kv = float(RNG.choice([131072.0, 163840.0, 262144.0]))
    beta = float(RNG.uniform(1.5, 4.0)) if backlog else float(RNG.uniform(0.05, 0.9))
    B = r_d * s_kv / beta
    return sch.Rates(r_p=r_p, r_d=r_d, B=B, s_kv=s_kv, T_load=float(RNG.uniform(0, 0.5)),
                     T_0=float(RNG.uniform(0.01, 0.3)), alpha=alpha, T_max=5.0, dT=dT)


def t_c(rt, K, T_rem):
    rho = rt.r_d / rt.r_p
    return (rt.T_load + (K + rt.r_d * T_rem) / rt.r_p) / (1 + rho)


def bracket(T, rt, T_limit):
    lo = math.floor(T / rt.dT) * rt.dT
    hi = min(lo + rt.dT, T_limit)
    return max(0.0, min(lo, T_limit)), hi


@pytest.mark.parametrize("trial", range(20))
def test_no_backlog_v_shape(trial):
    rt = random_rates(alpha=0.8)
    K, T_rem = float(RNG.uniform(200, 6000)), 20.0
    Tc = t_c(rt, K, T_rem)
    if not 0.1 < Tc < rt.T_max - 0.1:
        pytest.skip("T_c outside the window range for this draw")
    rho = rt.r_d / rt.r_p
    d = sch.select(rt, K, T_rem)

    def J(T):
        if T <= Tc:
            return rt.alpha * (rt.T_0 + (1 + rho) * (Tc - T))
        return rt.alpha * rt.T_0 + (1 - rt.alpha) * (1 + rho) * (T - Tc)

    lo, hi = bracket(Tc, rt, rt.T_max)
    want = min(J(lo), J(hi))
    assert d.best.J == pytest.approx(want, rel=1e-9, abs=1e-12)
    assert d.best.T_w == pytest.approx(lo if J(lo) <= J(hi) else hi, abs=1e-12)
    assert not d.trigger                      # T_remain = 20 s > any window: defer


@pytest.mark.parametrize("trial", range(10))
def test_alpha_one_first_window_past_tc(trial):
    rt = random_rates(alpha=1.0)
    K, T_rem = float(RNG.uniform(200, 6000)), 20.0
    Tc = t_c(rt, K, T_rem)
    if not 0.1 < Tc < rt.T_max - 0.1:
        pytest.skip("T_c outside the window range for this draw")
    d = sch.select(rt, K, T_rem)
    assert d.best.T_w == pytest.approx(math.ceil(Tc / rt.dT - 1e-9) * rt.dT, abs=1e-9)
    assert d.best.T_SIT == pytest.approx(rt.T_0, abs=1e-12)
    below = sch.evaluate(rt, K, T_rem, d.best.T_w - rt.dT)
    assert below.T_SIT > rt.T_0


def test_alpha_zero_selects_the_zero_window():
    rt = random_rates(alpha=0.0)
    d = sch.select(rt, 3000.0, 10.0)
    assert d.best.T_w == 0.0 and d.best.J == 0.0


@pytest.mark.parametrize("trial", range(10))
def test_backlog_crossing(trial):
    rt = random_rates(alpha=1.0, backlog=True)
    K, T_rem = float(RNG.uniform(200, 6000)), 20.0
    rho = rt.r_d / rt.r_p
    beta = rt.r_d * rt.s_kv / rt.B
    Tx = (1 + rho) * t_c(rt, K, T_rem) / (beta + rho)
    if not 0.1 < Tx < rt.T_max - 0.1:
        pytest.skip("crossing outside the window range for this draw")
    d = sch.select(rt, K, T_rem)

    def sit(T):
        return rt.T_0 + max((1 + rho) * (t_c(rt, K, T_rem) - T), (beta - 1) * T)

    lo, hi = bracket(Tx, rt, rt.T_max)
    assert d.best.T_SIT == pytest.approx(min(sit(lo), sit(hi)), rel=1e-9)
    assert d.best.T_SIT > rt.T_0            # a backlog always remains


def test_trigger_and_grid():
    rt = sch.Rates(r_p=8000.0, r_d=25.0, B=37.5e6, s_kv=262144.0, T_0=0.2, dT=0.2, T_max=5.0)
    assert len(sch.candidates(5.0, 0.2)) == 26             # 0, 0.2, ..., 5.0
    assert sch.candidates(0.5, 0.2)[-1] == 0.5 and len(sch.candidates(0.5, 0.2)) == 4
    assert sch.candidates(0.0, 0.2) == [0.0]
    far = sch.select(rt, 3000.0, 30.0)
    assert not far.trigger and far.n_candidates == 26
    # close to handover: T_limit = T_remain, and the chosen window reaches it
    near = sch.select(rt, 3000.0, 0.3)
    assert near.trigger and near.best.T_w <= 0.3
    # handover already passed: only the zero window, trigger at once
    late = sch.select(rt, 3000.0, -1.0)
    assert late.trigger and late.n_candidates == 1 and late.best.T_w == 0.0


def test_waste_bound_by_brute_force():
    """Eq. 10: preparation starts at most T_max + E_early before the actual
    handover, and work in its last T_avail seconds is useful; the wasted
    duration of every start time in that range stays under the bound, and
    the earliest start meets it."""
    for _ in range(200):
        T_max, E, A = RNG.uniform(0, 5), RNG.uniform(0, 4), RNG.uniform(0, 6)
        bound = sch.waste_bound(T_max, E, A)
        starts = np.linspace(0.0, T_max + E, 101)          # seconds before the handover
        waste = np.maximum(starts - A, 0.0)
        assert np.all(waste <= bound + 1e-12)
        assert waste[-1] == pytest.approx(bound)


def test_ewma_geometric():
    v = None
    for _ in range(1):
        v = sch.ewma(v, 10.0, 0.3)
    assert v == 10.0
    for k in range(1, 20):
        v = sch.ewma(v, 4.0, 0.3)
        assert v == pytest.approx(4.0 + 0.7 ** k * 6.0, rel=1e-12)


def test_admission():
    """The state expected at handover is the history the target would have
    to hold if preparation started at the last moment: Eq. 9's L_hist at a
    zero window (evaluate), as a KV cache (Eq. 1, footprint.cache_bytes).
    Admission holds exactly when the free VRAM covers that many bytes, and
    never for an incompatible model; a handover already due (T_remain <= 0)
    needs the current context only."""
    from oracle import footprint
    rt = sch.Rates(r_p=17500.0, r_d=25.0, B=300e6 / 8, s_kv=262144.0)
    for K_curr, T_remain in ((3000, 2.0), (4000, 0.0), (1234, -1.0), (10, 7.5)):
        L0 = sch.evaluate(rt, K_curr, max(T_remain, 0.0), 0.0).L_hist
        need = footprint.cache_bytes(1, 64, 8, 128, 2) * L0
        assert sch.admit(True, need, rt.s_kv, K_curr, rt.r_d, T_remain)
        assert not sch.admit(True, need - 1, rt.s_kv, K_curr, rt.r_d, T_remain)
        assert not sch.admit(False, 1e15, rt.s_kv, K_curr, rt.r_d, T_remain)
