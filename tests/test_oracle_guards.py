"""Pins of the oracle's calibration and rate guards (Section 5: calibration-
aware entropy, robust control with uncertainty floors, guard iii on the rate
of change of thresholds and temperatures, and the entropy-bias stress knob).

Each check is fixed independently of the oracle's formulas: the wrapper
identity of calibration (logits scaled by c and undone by T_cal = c give the
original distribution, entropy and samples), the rate bounds as inequalities
over random trajectories, the exact per-step descent of the kept fraction
after an entropy collapse, and the reduction of every guard to the unguarded
law at its neutral setting.
"""
import math

import numpy as np
import pytest

from oracle import blocks as Bk
from oracle import entropy as E
from oracle import sample as S
from synth import Params


def _params(**kw):
    base = dict(scale=0.125, eta=-0.05, h_target=2.5, t_min=0.05, t_max=5.0, eps_h=0.0,
                h_min=2.5, kappa_min=0.05, b_min=4, log_v=math.log(4096))
    base.update(kw)
    return Params(**base)


def test_neutral_settings_reduce_to_the_plain_law():
    rng = np.random.default_rng(0)
    p0 = _params()
    for _ in range(200):
        T = float(rng.uniform(0.05, 5.0))
        h = float(rng.uniform(0.0, 9.0))
        assert E.temperature_next(T, h, 2.5, -0.05, 0.05, 5.0, math.inf) == \
            E.temperature_next(T, h, 2.5, -0.05, 0.05, 5.0)
        kp = float(rng.uniform(0.0, 1.0))
        assert Bk.kept_fraction(h, p0, kp) == Bk.kept_fraction(h, p0)      # dkappa = 1
        assert Bk.keep_budget(h, 300, p0, kp) == Bk.keep_budget(h, 300, p0)
    z = rng.normal(0, 2.0, 4096)
    assert E.control_entropy(z, 0.7, p0) == E.entropy(z, 0.7)


@pytest.mark.parametrize("rho", [0.0, 0.01, 0.1, 0.5])
def test_temperature_rate_bound(rho):
    """|ln T_{t+1} - ln T_t| <= rho whenever no clip bound is hit; rho = 0
    freezes the temperature."""
    rng = np.random.default_rng(1)
    for _ in range(500):
        T = float(rng.uniform(0.2, 2.0))
        h = float(rng.uniform(0.0, 12.0))
        eta = float(rng.choice([-0.5, -0.05, 0.05, 0.5]))
        Tn = E.temperature_next(T, h, 2.5, eta, 0.05, 5.0, rho)
        free = E.temperature_next(T, h, 2.5, eta, 0.05, 5.0)
        if 0.05 < Tn < 5.0:
            assert abs(math.log(Tn) - math.log(T)) <= rho + 1e-12
        # The bound only ever shortens the step, in the same direction.
        assert abs(math.log(Tn / T)) <= abs(math.log(free / T)) + 1e-12
        assert (Tn - T) * (free - T) >= 0.0
        if rho == 0.0:
            assert Tn == T


def test_rate_bounded_loop_still_converges():
    """Closed loop on fixed logits with the stabilising gain: the bounded
    controller reaches |H - H*| < 1e-3, more slowly than the free one."""
    z = np.random.default_rng(2).normal(0.0, 3.0, 2048)
    steps = {}
    for rho in (math.inf, 0.02):
        T = 1.0
        for t in range(5000):
            h = E.entropy(z, T)
            if abs(h - 2.5) < 1e-3:
                steps[rho] = t
                break
            T = E.temperature_next(T, h, 2.5, -0.3, 0.05, 5.0, rho)
        assert rho in steps, rho
    assert steps[0.02] > steps[math.inf]


@pytest.mark.parametrize("dk", [0.05, 0.2])
def test_kept_fraction_descends_by_at_most_dkappa(dk):
    """After the entropy collapses from log|V| to 0 the kept fraction falls
    by exactly dkappa per step until it meets the unguarded value; a rise is
    immediate."""
    p = _params(dkappa=dk)
    f = np.float32
    kappa = Bk.kept_fraction(p.log_v, p)            # 1.0
    assert kappa == f(1.0)
    traj = [kappa]
    for _ in range(40):
        kappa = Bk.kept_fraction(0.0, p, kappa)
        traj.append(kappa)
    floor = Bk.kept_fraction(0.0, p)                 # kappa_min
    for a, b in zip(traj, traj[1:]):
        assert b == max(floor, f(a - f(dk)))
        assert b >= a - f(dk)
    assert traj[-1] == floor
    # Rise: back to log|V| in one step.
    assert Bk.kept_fraction(p.log_v, p, floor) == f(1.0)
    # The budget never falls below what the bounded fraction implies.
    for nb in (1, 7, 300):
        k_prev = Bk.keep_budget(p.log_v, nb, p)
        k_next = Bk.keep_budget(0.0, nb, p, 1.0)
        assert k_next >= min(k_prev, math.ceil((1.0 - dk) * nb) - 1)
    assert Bk.kept_fraction(0.0, p, math.nan) == floor


@pytest.mark.parametrize("c", [0.5, 2.0, 3.0])
def test_calibration_undoes_logit_scaling(c):
    """Miscalibration modelled as logits scaled by c (c > 1 overconfident,
    c < 1 underconfident); the calibration temperature T_cal = c restores
    the model's distribution: same entropy, same estimates, same samples."""
    rng = np.random.default_rng(3)
    z = rng.normal(0.0, 2.0, 3000)
    pc = _params(t_cal=c)
    for T in (0.5, 1.0, 2.0):
        assert abs(E.control_entropy(c * z, T, pc) - E.entropy(z, T)) < 1e-9
        for est in (E.TOPK, E.TAIL):
            pe, pce = _params(estimator=est, est_k=64), _params(estimator=est, est_k=64, t_cal=c)
            assert abs(E.control_entropy(c * z, T, pce) - E.control_entropy(z, T, pe)) < 1e-9
        for u in (0.0, 0.25, 0.7, 0.999):
            x1, m1 = S.sample(c * z, E.effective_temperature(T, pc), u)
            x0, m0 = S.sample(z, T, u)
            assert x1 == x0 or min(m0, m1) < 1e-9
    # Uncalibrated overconfidence lowers the entropy, and with it the budget.
    p = _params()
    if c > 1:
        assert E.control_entropy(c * z, 1.0, p) < E.entropy(z, 1.0)


@pytest.mark.parametrize("bias", [-1.5, 0.0, 0.75])
def test_entropy_bias_shifts_what_the_controller_sees(bias):
    rng = np.random.default_rng(4)
    z = rng.normal(0.0, 1.5, 4096)
    p = _params(h_bias=bias)
    h = E.entropy(z, 1.0)
    hc = E.control_entropy(z, 1.0, p)
    assert abs(hc - (h + bias)) < 1e-6
    assert Bk.keep_budget(hc, 500, _params()) == Bk.keep_budget(h + bias, 500, _params())
