"""Pins of the oracle's entropy-aware scheduler (Section 3.1 priority,
Section 7 bounded priority and no starvation).

Fixed independently of the oracle's code: the selection's defining
invariant (every selected sequence outranks every other, ties to the lower
index) over random and tied priorities; monotonicity of the priority in each
of its terms; the EWMA's closed-form convergence; bounded priorities; and a
pool simulation in which every sequence is served within a bounded wait.
"""
import math
from types import SimpleNamespace

import numpy as np
import pytest

from oracle import schedule as Sc


def _prm(**kw):
    base = dict(alpha=1.0, beta=0.25, gamma=4.0, slo=16.0, slack_floor=0.5, gain_floor=1e-3,
                ewma_rate=0.25)
    base.update(kw)
    return SimpleNamespace(**base)


@pytest.mark.parametrize("seed", range(4))
def test_selection_invariant(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 60))
    pri = rng.choice([0.1, 0.2, 0.3], size=n).astype(np.float32) if seed % 2 else \
        rng.random(n).astype(np.float32)
    for b in (0, 1, n // 2, n, n + 3):
        sel = Sc.select(pri, b)
        assert len(sel) == min(b, n)
        assert list(sel) == sorted(sel)
        rest = sorted(set(range(n)) - set(sel.tolist()))
        for s in sel:
            for r in rest:
                assert pri[s] > pri[r] or (pri[s] == pri[r] and s < r)


def test_priority_monotone_in_each_term():
    p = _prm()
    base = dict(gain=0.5, kept_blocks=100, ctx_len=3000, age=3)
    pi0 = Sc.priority(prm=p, **base)
    assert Sc.priority(prm=p, **{**base, "gain": 0.6}) > pi0
    assert Sc.priority(prm=p, **{**base, "kept_blocks": 120}) < pi0
    assert Sc.priority(prm=p, **{**base, "ctx_len": 4000}) < pi0
    assert Sc.priority(prm=p, **{**base, "age": 6}) > pi0
    # Past the slack floor, waiting longer changes nothing; below the gain
    # floor, the gain does not matter.
    assert Sc.priority(prm=p, **{**base, "age": 100}) == Sc.priority(prm=p, **{**base, "age": 200})
    assert Sc.priority(prm=p, **{**base, "gain": 0.0}) == Sc.priority(prm=p, **{**base, "gain": 1e-6})
    # Bounded: at most gain / (gamma * slack_floor), never below a positive floor.
    assert Sc.priority(prm=p, gain=10.0, kept_blocks=0, ctx_len=0, age=1000) <= \
        10.0 / (p.gamma * p.slack_floor) * (1 + 1e-6)
    assert Sc.priority(prm=p, gain=0.0, kept_blocks=10 ** 6, ctx_len=10 ** 8, age=0) > 0


@pytest.mark.parametrize("lam", [1.0, 0.5, 0.1])
def test_ewma_converges_geometrically(lam):
    g, tl, tau = np.float32(2.0), np.float32(0.0), 0.0
    d = 0.3
    for t in range(1, 40):
        tau += d
        g, tl = Sc.update_gain(g, tau, tl, True, lam)
        assert abs(g - d) <= abs(2.0 - d) * (1 - lam) ** t + 1e-5
    assert abs(g - d) < 1e-3 or lam == 0.1
    # A sequence that did not run keeps its mean and its mark.
    g2, tl2 = Sc.update_gain(g, tau + 5.0, tl, False, lam)
    assert g2 == g and tl2 == tl


def test_no_starvation_in_a_pool():
    """Section 7's no-starvation argument: sequences that keep running resolve
    (their entropy drops shrink), their priority falls, and the others are
    served.  64 sequences with fixed, very unequal costs, 8 served per step,
    each run's entropy drop shrinking by 5%: every sequence is served, and
    the most expensive sequence is served once the cheap ones resolve."""
    rng = np.random.default_rng(7)
    n, b = 64, 8
    p = _prm(slo=24.0)
    kept = rng.integers(10, 2000, n)
    ctx = rng.integers(100, 60000, n)
    d0 = rng.uniform(0.05, 0.6, n)
    runs = np.zeros(n, dtype=np.int64)
    tau = np.zeros(n, dtype=np.float32)
    tau_last = np.zeros(n, dtype=np.float32)
    gain = np.full(n, 1.0, dtype=np.float32)
    age = np.zeros(n, dtype=np.int32)
    first = np.full(n, -1)
    for step in range(600):
        sel, pri, tau_last, gain, age = Sc.schedule(tau, tau_last, gain, age, kept, ctx, b, p)
        assert np.all(np.isfinite(pri)) and np.all(pri > 0)
        for s in sel:
            if first[s] < 0:
                first[s] = step
            tau[s] += np.float32(d0[s] * 0.95 ** runs[s])            # the sequence runs
            runs[s] += 1
    assert np.all(first >= 0), np.nonzero(first < 0)[0]
    costly = int(np.argmax(1.0 * kept + 0.25 * ((ctx + 15) // 16)))
    assert first[costly] > 0
