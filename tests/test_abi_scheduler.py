"""The library's host-side Scheduler Engine (pallas_window_*, pallas_ewma_update,
pallas_admit, pallas_waste_bound) against the oracle's, on seeded sweeps of
rates, contexts and remaining times: the same window, cost, interruption
and trigger decision, the same smoothing, admission and bound.  No GPU."""
import numpy as np
import pytest

from helpers import ensure_lib
from oracle import scheduler as sch


@pytest.fixture(scope="module")
def P():
    return ensure_lib()


def draw(rng):
    beta = rng.uniform(0.05, 4.0)
    r_d = rng.uniform(1, 100)
    s_kv = rng.choice([1024.0, 147456.0, 262144.0])
    return dict(r_p=rng.uniform(100, 40000), r_d=r_d, goodput=r_d * s_kv / beta, s_kv=s_kv,
                t_load=rng.choice([0.0, rng.uniform(0, 2)]), t_0=rng.uniform(0, 0.5),
                alpha=rng.choice([0.0, 0.8, 1.0, rng.uniform(0, 1)]), t_max=rng.choice([0.0, 2.0, 5.0, 7.3]),
                dt=rng.choice([0.2, 0.05, 0.013]))


def rates(p):
    return sch.Rates(r_p=p["r_p"], r_d=p["r_d"], B=p["goodput"], s_kv=p["s_kv"], T_load=p["t_load"],
                     T_0=p["t_0"], alpha=p["alpha"], T_max=p["t_max"], dT=p["dt"])


@pytest.mark.parametrize("seed", range(8))
def test_window_select_matches_oracle(P, seed):
    rng = np.random.default_rng(seed)
    for _ in range(60):
        p = draw(rng)
        K = float(rng.uniform(0, 9000))
        T_rem = float(rng.choice([rng.uniform(-1, 0), rng.uniform(0, 1), rng.uniform(1, 12)]))
        d = P.pallas_window_select(K, T_rem, **p)
        o = sch.select(rates(p), K, T_rem)
        assert d.n_candidates == o.n_candidates
        assert bool(d.trigger) == o.trigger
        assert d.t_w == pytest.approx(o.best.T_w, rel=1e-12, abs=1e-12)
        for a, b in ((d.cost, o.best.J), (d.t_sit, o.best.T_SIT), (d.t_early, o.best.T_early),
                     (d.t_hist, o.best.T_hist), (d.t_res, o.best.T_res), (d.l_hist, o.best.L_hist)):
            assert a == pytest.approx(b, rel=1e-12, abs=1e-12)


def test_window_evaluate_matches_oracle(P):
    rng = np.random.default_rng(99)
    for _ in range(200):
        p = draw(rng)
        K, T_rem, T_w = float(rng.uniform(0, 9000)), float(rng.uniform(0, 10)), float(rng.uniform(0, 6))
        d = P.pallas_window_evaluate(K, T_rem, T_w, **p)
        o = sch.evaluate(rates(p), K, T_rem, T_w)
        assert d.cost == pytest.approx(o.J, rel=1e-12, abs=1e-12)
        assert d.t_sit == pytest.approx(o.T_SIT, rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("bad", [dict(r_p=0.0), dict(goodput=-1.0), dict(dt=0.0), dict(alpha=1.5),
                                 dict(t_max=-1.0), dict(r_d=float("nan")), dict(t_max=1e9, dt=1e-3)])
def test_window_rejects_bad_parameters(P, bad):
    p = dict(r_p=8000.0, r_d=25.0, goodput=37.5e6, s_kv=262144.0, t_0=0.1)
    p.update(bad)
    with pytest.raises(P.PallasError) as e:
        P.pallas_window_select(3000.0, 1e9, **p)
    assert e.value.status == P.Status.INVALID_ARG


def test_ewma_admit_and_bound_match_oracle(P):
    rng = np.random.default_rng(5)
    st, ref = P.Ewma(), None
    for _ in range(50):
        x, w = float(rng.uniform(0, 1e4)), 0.25
        assert P.pallas_ewma_update(st, x, w) == pytest.approx(sch.ewma(ref, x, w), rel=1e-15)
        ref = sch.ewma(ref, x, w)
    assert np.isnan(P.pallas_ewma_update(st, 1.0, 0.0))
    for _ in range(100):
        args = (bool(rng.integers(0, 2)), float(rng.uniform(0, 3e9)), 262144.0,
                float(rng.uniform(0, 9000)), float(rng.uniform(0, 100)), float(rng.uniform(-1, 10)))
        assert P.pallas_admit(*args) == sch.admit(*args)
        t = [float(v) for v in rng.uniform(0, 6, 3)]
        assert P.pallas_waste_bound(*t) == sch.waste_bound(*t)
