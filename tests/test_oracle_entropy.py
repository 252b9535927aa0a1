"""Pins of the oracle's entropy, entropic time and temperature law.

Each check is fixed by mathematics independent of the oracle's own code:
closed forms, invariances, a library routine, a derivative identity, and the
stability properties the paper states for the controller (Section 7,
Proposition 1; Appendix A, the ISS theorem).
"""
import math

import numpy as np
import pytest
import scipy.stats

from oracle import entropy as E
from synth import Params


def _params(**kw):
    base = dict(scale=0.125, eta=-0.05, h_target=2.5, t_min=0.05, t_max=5.0, eps_h=0.0,
                h_min=2.5, kappa_min=0.05, b_min=4, log_v=math.log(1024))
    base.update(kw)
    return Params(**base)


@pytest.mark.parametrize("V", [1, 2, 7, 1024, 128256])
@pytest.mark.parametrize("T", [0.05, 1.0, 3.7])
def test_uniform_is_log_v(V, T):
    z = np.full(V, 0.37)
    assert abs(E.entropy(z, T) - math.log(V)) < 1e-12


def test_one_hot_is_zero():
    z = np.zeros(4096)
    z[17] = 1000.0
    assert E.entropy(z, 1.0) == 0.0
    z = np.full(100, -np.inf)
    z[3] = 2.0
    assert E.entropy(z, 0.7) == 0.0


@pytest.mark.parametrize("k", [1, 2, 3, 10, 777])
def test_tied_maxima_is_log_k(k):
    rng = np.random.default_rng(k)
    z = np.full(2000, -np.inf)
    z[rng.choice(2000, size=k, replace=False)] = 5.5
    assert abs(E.entropy(z, 1.3) - math.log(k)) < 1e-12


@pytest.mark.parametrize("a,b", [(0.0, 0.0), (1.0, -2.0), (-3.5, 4.25), (20.0, 0.0)])
def test_two_logits_binary_entropy(a, b):
    p = 1.0 / (1.0 + math.exp(b - a))
    hb = -(p * math.log(p) + (1 - p) * math.log(1 - p))
    assert abs(E.entropy(np.array([a, b]), 1.0) - hb) < 1e-12


def test_shift_permutation_and_temperature_invariance():
    rng = np.random.default_rng(1)
    z = rng.normal(0, 2.5, 5000)
    h = E.entropy(z, 1.7)
    assert abs(E.entropy(z + 123.25, 1.7) - h) < 1e-10
    assert abs(E.entropy(rng.permutation(z), 1.7) - h) < 1e-10
    assert abs(E.entropy(z / 1.7, 1.0) - h) < 1e-10


@pytest.mark.parametrize("seed", range(5))
def test_matches_scipy_entropy(seed):
    rng = np.random.default_rng(seed)
    z = rng.normal(0, rng.uniform(0.3, 6), 3000)
    T = rng.uniform(0.2, 3)
    w = np.exp(z / T - np.max(z / T))
    assert abs(E.entropy(z, T) - scipy.stats.entropy(w)) < 1e-10


@pytest.mark.parametrize("T", [0.3, 1.0, 2.5])
def test_log_temperature_derivative_is_variance(T):
    # For p proportional to exp(z/T): dH/dlog T = Var_p(z/T) >= 0.
    rng = np.random.default_rng(7)
    z = rng.normal(0, 2.0, 4000)
    eps = 1e-5
    num = (E.entropy(z, T * math.exp(eps)) - E.entropy(z, T * math.exp(-eps))) / (2 * eps)
    y = z / T
    p = np.exp(y - y.max())
    p /= p.sum()
    var = float(np.sum(p * y * y) - np.sum(p * y) ** 2)
    assert var > 0
    assert abs(num - var) < 1e-5 * max(1.0, var)


def test_small_spread_asymptote():
    # H = log V - Var(z)/2 + O(s^3) for logits of small spread s.
    rng = np.random.default_rng(3)
    z = rng.normal(0, 0.02, 128256)
    pred = math.log(128256) - np.var(z) / 2
    assert abs(E.entropy(z, 1.0) - pred) < 1e-5


def test_entropic_time_closed_forms():
    assert E.entropic_time(1.0, 3.0, 2.0) == 2.0
    assert E.entropic_time(1.0, 2.0, 3.0) == 1.0
    assert E.entropic_time(0.5, math.nan, 9.0) == 0.5
    rng = np.random.default_rng(0)
    hs = rng.uniform(0, 10, 200)
    tau, prev = 0.0, math.nan
    taus = []
    for h in hs:
        tau = E.entropic_time(tau, prev, h)
        prev = h
        taus.append(tau)
    assert np.all(np.diff(taus) >= 0)
    # Telescoping for a nonincreasing sequence, zero for a nondecreasing one.
    down = np.sort(hs)[::-1]
    tau, prev = 0.0, math.nan
    for h in down:
        tau, prev = E.entropic_time(tau, prev, h), h
    assert abs(tau - (down[0] - down[-1])) < 1e-9
    tau, prev = 0.0, math.nan
    for h in np.sort(hs):
        tau, prev = E.entropic_time(tau, prev, h), h
    assert tau == 0.0


def test_temperature_fixed_at_target():
    for T in (0.05, 0.731, 1.0, 4.99):
        assert E.temperature_next(T, 2.5, 2.5, -0.05, 0.05, 5.0) == T
        assert E.temperature_next(T, 2.5, 2.5, +0.05, 0.05, 5.0) == T


def test_temperature_closed_form_direction_and_clip():
    assert abs(E.temperature_next(1.0, 4.5, 2.5, -0.05, 0.05, 5.0) - math.exp(-0.1)) < 1e-15
    assert abs(E.temperature_next(2.0, 0.5, 2.5, -0.05, 0.05, 5.0) - 2.0 * math.exp(0.1)) < 1e-15
    assert E.temperature_next(4.9, 0.0, 2.5, -1.0, 0.05, 5.0) == 5.0
    assert E.temperature_next(0.06, 11.0, 2.5, -1.0, 0.05, 5.0) == 0.05
    # Stabilising sign: above the target the temperature falls, below it rises.
    assert E.temperature_next(1.0, 3.0, 2.5, -0.05, 0.05, 5.0) < 1.0
    assert E.temperature_next(1.0, 2.0, 2.5, -0.05, 0.05, 5.0) > 1.0


def _loop(z, T, params, steps, noise=None):
    Ts, Hs = [], []
    for t in range(steps):
        h = E.entropy(z, T)
        Hs.append(h)
        hm = h + (0.0 if noise is None else noise[t])
        T = E.temperature_next(T, hm, params.h_target, params.eta, params.t_min, params.t_max)
        Ts.append(T)
    return np.array(Ts), np.array(Hs)


def test_closed_loop_converges_with_stabilising_gain():
    rng = np.random.default_rng(11)
    z = rng.normal(0, 2.0, 4096)
    p = _params()
    Ts, Hs = _loop(z, 1.0, p, 400)
    assert abs(Hs[-1] - p.h_target) < 1e-3
    assert np.all((Ts >= p.t_min) & (Ts <= p.t_max))


def test_printed_positive_gain_runs_to_a_clip_bound():
    # The law with the printed positive gain is positive feedback for a
    # softmax: the temperature leaves the target and ends on a clip bound.
    rng = np.random.default_rng(11)
    z = rng.normal(0, 2.0, 4096)
    p = _params(eta=0.05)
    Ts, Hs = _loop(z, 1.0, p, 400)
    assert Ts[-1] in (p.t_min, p.t_max)
    assert abs(Hs[-1] - p.h_target) > 1.0


def _t_star(z, h_target):
    lo, hi = 1e-3, 1e3
    for _ in range(200):
        mid = math.sqrt(lo * hi)
        if E.entropy(z, mid) < h_target:
            lo = mid
        else:
            hi = mid
    return math.sqrt(lo * hi)


def test_iss_bound_under_bounded_estimator_noise():
    # Appendix A: with |e_t| <= eps_H and restoring slope mu on the
    # neighbourhood, |log T_t - log T*| <= a^t |delta_0| + eps_H / mu,
    # a = 1 - |eta| mu (with the stabilising sign of the gain).
    rng = np.random.default_rng(5)
    z = rng.normal(0, 2.0, 4096)
    p = _params(eta=-0.2)
    Tstar = _t_star(z, p.h_target)
    r = 0.6
    grid = np.linspace(-r, r, 121)
    slopes = []
    for d in grid:
        T = Tstar * math.exp(d)
        y = z / T
        q = np.exp(y - y.max())
        q /= q.sum()
        slopes.append(float(np.sum(q * y * y) - np.sum(q * y) ** 2))
    mu, mu_max = min(slopes), max(slopes)
    eta = abs(p.eta)
    assert 0 < eta * mu < 1 and eta * mu_max < 1
    a = 1 - eta * mu
    eps_h = 0.02
    noise = rng.uniform(-eps_h, eps_h, 300)
    T0 = Tstar * math.exp(0.5)
    Ts, _ = _loop(z, T0, p, 300, noise)
    delta0 = abs(math.log(T0 / Tstar))
    for t, T in enumerate(Ts, start=1):
        assert abs(math.log(T / Tstar)) <= a ** t * delta0 + eps_h / mu + 1e-9


def test_control_step_batch():
    rng = np.random.default_rng(2)
    z = rng.normal(0, 2, (3, 500))
    p = _params()
    out = E.control_step(z, np.array([np.nan, 10.0, 0.0]), np.array([0.0, 1.0, 2.0]),
                         np.array([1.0, 0.5, 2.0]), p)
    for b in range(3):
        h = E.entropy(z[b], [1.0, 0.5, 2.0][b])
        assert out["h"][b] == h
    assert out["tau"][0] == 0.0
    assert abs(out["tau"][1] - (1.0 + 10.0 - out["h"][1])) < 1e-12
    assert out["tau"][2] == 2.0
    assert list(out["temp_used"]) == [1.0, 0.5, 2.0]
