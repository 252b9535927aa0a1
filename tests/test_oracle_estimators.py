"""Pins of the oracle's top-k and tail-corrected entropy estimators.

Each check is fixed by mathematics independent of the oracle's code: the
top-k set as the k-subset of largest probability mass (brute force over all
subsets), the grouping rule of Shannon entropy, the bounds the paper states
for both estimators (Section 2.1), closed forms for two-token and one-token
cases, uniform tails (where the tail term is exact), and the conservative
direction of the guarded budget (Section 3.3).
"""
import itertools
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats

from oracle import blocks as Bk
from oracle import entropy as E
from synth import Params


def _params(**kw):
    base = dict(scale=0.125, eta=-0.05, h_target=2.5, t_min=0.05, t_max=5.0, eps_h=0.0,
                h_min=2.5, kappa_min=0.05, b_min=4, log_v=math.log(4096))
    base.update(kw)
    return Params(**base)


def _rows(seed=0):
    """Logit rows of several shapes: Gaussian of small and large spread, Zipf
    ranks at a random position, heavy ties, masked entries."""
    rng = np.random.default_rng(seed)
    out = []
    for V in (9, 257, 4096):
        for s in (0.3, 1.0, 4.0):
            out.append(rng.normal(0.0, s, V))
        r = rng.permutation(V) + 1
        out.append(-1.2 * np.log(r))
        out.append(rng.integers(0, 4, V).astype(np.float64))        # ties at every level
        z = rng.normal(0.0, 2.0, V)
        z[rng.random(V) < 0.5] = -np.inf
        z[0] = 1.0
        out.append(z)
    return out


def _softmax(z, T):
    return scipy.special.softmax(np.asarray(z, dtype=np.float64) / T)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_topk_is_the_heaviest_subset(seed):
    """The top-k set is the k-subset of largest total probability; every such
    subset (ties) gives the same H~ and m.  Brute force over all subsets."""
    rng = np.random.default_rng(seed)
    V = 7
    z = rng.normal(0.0, 1.5, V)
    z[2] = z[5]                                  # a tie
    T = 0.8
    p = _softmax(z, T)
    for k in range(1, V + 1):
        best = max(p[list(S)].sum() for S in itertools.combinations(range(V), k))
        heaviest = [S for S in itertools.combinations(range(V), k)
                    if abs(p[list(S)].sum() - best) < 1e-15]
        ht, m, mbar = E.topk_entropy(z, T, k)
        assert abs(m - best) < 1e-13
        assert abs(mbar - (1.0 - best)) < 1e-13
        for S in heaviest:
            assert abs(ht - scipy.stats.entropy(p[list(S)])) < 1e-12


@pytest.mark.parametrize("k", [1, 4, 64, 256, 4095, 4096, 10 ** 6])
@pytest.mark.parametrize("T", [0.3, 1.0, 2.5])
def test_estimators_bracket_the_entropy(k, T):
    """H~ <= H <= H^ when K is the top-k set (Section 2.1: H~ is the lower
    bound, the uniform-tail expression the upper bound)."""
    for z in _rows():
        H = E.entropy(z, T)
        ht, _, _ = E.topk_entropy(z, T, k)
        hh = E.tail_corrected_entropy(z, T, k)
        assert ht <= H + 1e-12
        assert H <= hh + 1e-12


@pytest.mark.parametrize("k", [1, 3, 50, 256])
def test_grouping_rule(k):
    """H = m H~ + h(mbar) + mbar H_tail, with H_tail the entropy of the
    renormalised tail (grouping property of Shannon entropy)."""
    T = 1.3
    for z in _rows(5):
        p = np.sort(_softmax(z, T))[::-1]
        kk = min(k, p.size)
        ht, m, mbar = E.topk_entropy(z, T, k)
        tail = p[kk:]
        h_tail = scipy.stats.entropy(tail) if tail.sum() > 0 else 0.0
        rhs = m * ht + E.binary_entropy(mbar) + mbar * h_tail
        assert abs(E.entropy(z, T) - rhs) < 1e-10


@pytest.mark.parametrize("V,k", [(10, 3), (4096, 256), (128256, 64)])
def test_uniform_tail_gap(V, k):
    """With a uniform tail the bound's only slack is the top-k term:
    H^ - H = mbar H~ exactly (grouping rule with H_tail = ln(|V| - k))."""
    rng = np.random.default_rng(V)
    z = np.full(V, -1.0)
    z[rng.choice(V, k, replace=False)] = rng.uniform(-0.5, 3.0, k)  # k distinct values above
    for T in (0.7, 1.0, 3.0):
        ht, _, mbar = E.topk_entropy(z, T, k)
        gap = E.tail_corrected_entropy(z, T, k) - E.entropy(z, T)
        assert abs(gap - mbar * ht) < 1e-10
        assert gap <= mbar * (ht + math.log(V - k)) + 1e-12


@pytest.mark.parametrize("T", [0.2, 1.0])
def test_no_tail_is_exact(T):
    """k >= |V|, or a row with only k finite logits: mbar = 0 and both
    estimators equal the exact entropy."""
    rng = np.random.default_rng(3)
    z = rng.normal(0.0, 2.0, 300)
    H = E.entropy(z, T)
    for k in (300, 301, 5000):
        assert E.topk_entropy(z, T, k)[2] == 0.0
        assert abs(E.topk_entropy(z, T, k)[0] - H) < 1e-12
        assert abs(E.tail_corrected_entropy(z, T, k) - H) < 1e-12
    z2 = np.full(300, -np.inf)
    z2[rng.choice(300, 17, replace=False)] = rng.normal(0.0, 1.0, 17)
    H2 = E.entropy(z2, T)
    assert abs(E.topk_entropy(z2, T, 17)[0] - H2) < 1e-12
    assert abs(E.tail_corrected_entropy(z2, T, 17) - H2) < 1e-12


@pytest.mark.parametrize("a,b", [(0.0, 0.0), (1.0, -2.0), (5.0, 4.9), (-3.0, 7.0)])
def test_two_tokens_k1(a, b):
    """|V| = 2, k = 1: H~ = 0 and H^ = h(mbar) = the exact entropy, the binary
    entropy of the logistic probability."""
    z = np.array([a, b])
    pb = 1.0 / (1.0 + math.exp(-abs(a - b)))        # larger probability
    q = 1.0 - pb
    hb = -pb * math.log(pb) - (q * math.log(q) if q > 0 else 0.0)
    assert abs(E.topk_entropy(z, 1.0, 1)[0]) < 1e-14
    assert abs(E.tail_corrected_entropy(z, 1.0, 1) - hb) < 1e-12
    assert abs(E.entropy(z, 1.0) - hb) < 1e-12


def test_k1_closed_form():
    """k = 1: H~ = 0; H^ = h(1 - p_max) + (1 - p_max) ln(|V| - 1)."""
    rng = np.random.default_rng(9)
    for V in (5, 1000):
        z = rng.normal(0.0, 1.0, V)
        pmax = _softmax(z, 1.0).max()
        q = 1.0 - pmax
        want = -q * math.log(q) - pmax * math.log(pmax) + q * math.log(V - 1)
        assert abs(E.topk_entropy(z, 1.0, 1)[0]) < 1e-14
        assert abs(E.tail_corrected_entropy(z, 1.0, 1) - want) < 1e-12


def test_invariances():
    """Shift, permutation and temperature invariances carry over from p."""
    rng = np.random.default_rng(4)
    z = rng.normal(0.0, 1.5, 2000)
    for k in (1, 20, 700):
        for f in (lambda x, T: E.topk_entropy(x, T, k)[0],
                  lambda x, T: E.tail_corrected_entropy(x, T, k)):
            ref = f(z, 1.7)
            assert abs(f(z + 123.0, 1.7) - ref) < 1e-10
            assert abs(f(rng.permutation(z), 1.7) - ref) < 1e-12
            assert abs(f(z / 1.7, 1.0) - ref) < 1e-12


def test_estimate_dispatch():
    z = np.random.default_rng(0).normal(0.0, 1.0, 500)
    assert E.entropy_estimate(z, 1.0) == E.entropy(z, 1.0)
    assert E.entropy_estimate(z, 1.0, E.TOPK, 10) == E.topk_entropy(z, 1.0, 10)[0]
    assert E.entropy_estimate(z, 1.0, E.TAIL, 10) == E.tail_corrected_entropy(z, 1.0, 10)
    with pytest.raises(ValueError):
        E.entropy_estimate(z, 1.0, 7, 10)


def test_guarded_budget_is_conservative():
    """Section 3.3 guard: the budget is evaluated at H_g = max(H^ + eps_H,
    H_min).  The tail-corrected estimate never prunes more than the exact
    entropy would; the top-k estimate can, unless eps_H covers its gap
    h(mbar) + mbar ln(|V| - k) (the bound H - H~ <= h(mbar) + mbar ln(|V| - k)
    follows from the grouping rule)."""
    V = 4096
    prm = _params(h_min=0.5, log_v=math.log(V))
    fewer_topk = 0
    for z in _rows(11):
        if z.size != V:
            continue
        for T in (0.5, 1.0, 2.0):
            H = E.entropy(z, T)
            for kk in (4, 64, 512):
                ht, _, mbar = E.topk_entropy(z, T, kk)
                hh = E.tail_corrected_entropy(z, T, kk)
                cert = E.binary_entropy(mbar) + mbar * math.log(V - kk)
                assert H - ht <= cert + 1e-12
                for nb in (7, 100, 512):
                    k_exact = Bk.keep_budget(H, nb, prm)
                    assert Bk.keep_budget(hh, nb, prm) >= k_exact
                    assert Bk.keep_budget(ht, nb, prm.replace(eps_h=cert + 1e-6)) >= k_exact
                    fewer_topk += Bk.keep_budget(ht, nb, prm) < k_exact
    assert fewer_topk > 0          # without the guard, top-k pruning is more aggressive


def test_controller_direction_with_tail_estimate():
    """With a stabilising gain the controller driven by H^ >= H lowers the
    temperature at least as much as the exact controller."""
    rng = np.random.default_rng(2)
    B, V = 8, 4096
    logits = rng.normal(0.0, 1.0, (B, V)) * rng.uniform(0.5, 4.0, (B, 1))
    hp = np.full(B, np.nan)
    tau = np.zeros(B)
    temp = rng.uniform(0.5, 2.0, B)
    pr = _params(log_v=math.log(V))
    ex = E.control_step(logits, hp, tau, temp, pr)
    tl = E.control_step(logits, hp, tau, temp, pr.replace(estimator=E.TAIL, est_k=32))
    assert np.all(tl["h"] >= ex["h"] - 1e-12)
    assert np.all(tl["temp_next"] <= ex["temp_next"] + 1e-15)
