"""Pins of the oracle's sampler: closed forms, monotonicity and a chi-square
frequency test against softmax(z / T)."""
import math

import numpy as np
import pytest
import scipy.stats

from oracle import sample as Sm


def test_one_hot_always_returns_the_hot_token():
    z = np.full(1024, -np.inf)
    z[613] = 0.0
    for u in (0.0, 1e-9, 0.5, 0.999999):
        assert Sm.sample(z, 0.8, u)[0] == 613
    z = np.zeros(1024)
    z[5] = 2000.0
    assert Sm.sample(z, 1.0, 0.3)[0] == 5


def test_u_zero_gives_first_positive_mass_token():
    z = np.full(100, -np.inf)
    z[[7, 50, 80]] = [1.0, 3.0, 2.0]
    assert Sm.sample(z, 1.0, 0.0)[0] == 7
    z = np.random.default_rng(0).normal(size=300)
    assert Sm.sample(z, 1.0, 0.0)[0] == 0


def test_monotone_in_u_and_interval_contains_u():
    rng = np.random.default_rng(1)
    z = rng.normal(0, 2, 5000)
    us = np.sort(rng.random(300))
    xs = [Sm.sample(z, 1.3, u)[0] for u in us]
    assert all(a <= b for a, b in zip(xs, xs[1:]))
    for u, x in zip(us[:40], xs[:40]):
        lo, hi = Sm.cdf_interval(z, 1.3, x)
        assert lo <= u < hi
    assert np.array_equal(Sm.sample_many(z, 1.3, us), xs)


def test_last_positive_mass_when_u_rounds_to_the_top():
    z = np.array([0.0, 1.0, -np.inf, -np.inf])
    x, _ = Sm.sample(z, 1.0, 1.0)     # u*S == S: no j with C_j > u*S
    assert x == 1


@pytest.mark.parametrize("T", [0.5, 1.0, 2.0])
def test_chi_square_frequencies(T):
    rng = np.random.default_rng(42)
    z = rng.normal(0, 1.5, 1024)
    us = rng.random(100_000)
    xs = Sm.sample_many(z, T, us)
    y = z / T
    p = np.exp(y - y.max())
    p /= p.sum()
    counts = np.bincount(xs, minlength=1024).astype(float)
    exp = p * len(us)
    # merge tokens with small expected counts into one bin
    big = exp >= 5
    obs = np.concatenate([counts[big], [counts[~big].sum()]])
    ex = np.concatenate([exp[big], [exp[~big].sum()]])
    if ex[-1] == 0:
        obs, ex = obs[:-1], ex[:-1]
    stat, pval = scipy.stats.chisquare(obs, ex)
    assert pval > 1e-3


def test_margin_is_distance_to_interval_edges():
    z = np.log(np.array([1.0, 2.0, 1.0]))   # probabilities 1/4, 1/2, 1/4
    x, r = Sm.sample(z, 1.0, 0.3)
    assert x == 1 and abs(r - 0.05) < 1e-12
    x, r = Sm.sample(z, 1.0, 0.74)
    assert x == 1 and abs(r - 0.01) < 1e-12
