"""Pins of the oracle's block summaries, block scores, budget and kept set.

The block-score reading has no printed values to compare against (parity
unpinned against the paper); what is pinned here is that the oracle computes
that reading correctly: a token-level brute force, closed forms (zero query,
identical blocks), the entropy identity the reading implies, and the budget
rule's limits.
"""
import math

import numpy as np
import pytest
import scipy.stats

from oracle import blocks as Bk
from synth import Params


def _params(**kw):
    base = dict(scale=0.125, eta=-0.05, h_target=2.5, t_min=0.05, t_max=5.0, eps_h=0.0,
                h_min=2.5, kappa_min=0.05, b_min=4, log_v=float(np.float32(math.log(128256))))
    base.update(kw)
    return Params(**base)


def test_block_token_counts():
    assert list(Bk.block_token_counts(0, 16)) == []
    assert list(Bk.block_token_counts(1, 16)) == [1]
    assert list(Bk.block_token_counts(16, 16)) == [16]
    assert list(Bk.block_token_counts(17, 16)) == [16, 1]
    assert list(Bk.block_token_counts(40, 16)) == [16, 16, 8]


def test_block_means_brute_force():
    rng = np.random.default_rng(0)
    K = rng.normal(size=(37, 3, 5))
    m = Bk.block_means(K, 16)
    assert m.shape == (3, 3, 5)
    for b, (lo, hi) in enumerate([(0, 16), (16, 32), (32, 37)]):
        for g in range(3):
            for j in range(5):
                ref = sum(K[i, g, j] for i in range(lo, hi)) / (hi - lo)
                assert abs(m[b, g, j] - ref) < 1e-12


def _token_level_scores(q, kbar, counts, scale):
    """Brute force: expand blocks to tokens carrying their block's mean key,
    take each head's softmax over tokens, and sum -a log a per block."""
    Hq = q.shape[0]
    Hkv = kbar.shape[1]
    G = Hq // Hkv
    out = np.zeros(len(counts))
    for h in range(Hq):
        logits = []
        owner = []
        for b, n in enumerate(counts):
            zb = scale * sum(q[h, j] * kbar[b, h // G, j] for j in range(q.shape[1]))
            logits += [zb] * int(n)
            owner += [b] * int(n)
        m = max(logits)
        w = [math.exp(x - m) for x in logits]
        tot = sum(w)
        for x, b in zip(w, owner):
            a = x / tot
            out[b] += -a * math.log(a) / Hq
    return out


@pytest.mark.parametrize("G", [1, 2, 4])
def test_scores_match_token_level_brute_force(G):
    rng = np.random.default_rng(G)
    Hkv, d = 2, 8
    q = rng.normal(size=(Hkv * G, d))
    counts = np.array([16, 16, 16, 5])
    kbar = rng.normal(size=(4, Hkv, d))
    I, I_h, z = Bk.block_scores(q, kbar, counts, 0.4)
    ref = _token_level_scores(q, kbar, counts, 0.4)
    assert np.allclose(I, ref, rtol=1e-12, atol=1e-14)


def test_zero_query_gives_uniform_attention_closed_form():
    rng = np.random.default_rng(1)
    counts = np.array([16] * 9 + [3])
    N = counts.sum()
    kbar = rng.normal(size=(10, 4, 16))
    I, I_h, _ = Bk.block_scores(np.zeros((8, 16)), kbar, counts, 0.25)
    assert np.allclose(I, counts / N * math.log(N), rtol=1e-13)


def test_head_scores_sum_to_attention_entropy():
    rng = np.random.default_rng(2)
    counts = np.array([16] * 30 + [7])
    kbar = rng.normal(size=(31, 2, 32))
    q = rng.normal(size=(4, 32)) * 2
    I, I_h, z = Bk.block_scores(q, kbar, counts, 1 / math.sqrt(32))
    N = counts.sum()
    for h in range(4):
        tok = np.repeat(z[:, h], counts)
        w = np.exp(tok - tok.max())
        Hh = scipy.stats.entropy(w)
        assert abs(I_h[:, h].sum() - Hh) < 1e-10
        assert I_h[:, h].sum() <= math.log(N) + 1e-12
    assert np.all(I >= 0)


def test_identical_blocks_score_equally_and_gqa_mapping():
    rng = np.random.default_rng(3)
    kb = rng.normal(size=(2, 16))
    kbar = np.stack([kb, kb, rng.normal(size=(2, 16)), kb])
    q = rng.normal(size=(4, 16))
    I, _, z = Bk.block_scores(q, kbar, np.array([16, 16, 16, 16]), 0.25)
    assert I[0] == I[1] == I[3]
    # head h reads KV head h // G (G = 2)
    for h in range(4):
        assert abs(z[2, h] - 0.25 * float(q[h] @ kbar[2, h // 2])) < 1e-12


def test_exact_diagnostic_equals_mean_key_reading_when_blocks_are_constant():
    rng = np.random.default_rng(4)
    N, Hkv, d, bs = 53, 2, 8, 16
    kb = rng.normal(size=(4, Hkv, d))
    K = np.repeat(kb, bs, axis=0)[:N]
    q = rng.normal(size=(4, d))
    counts = Bk.block_token_counts(N, bs)
    I, _, _ = Bk.block_scores(q, Bk.block_means(K, bs), counts, 0.3)
    Ie = Bk.exact_token_scores(q, K, bs, 0.3)
    assert np.allclose(I, Ie, rtol=1e-12, atol=1e-15)


def test_budget_limits():
    p = _params()
    for nb in (1, 3, 4, 5, 17, 512, 8192):
        assert Bk.keep_budget(p.log_v, nb, p) == nb
        assert Bk.keep_budget(50.0, nb, p) == nb
        low = max(min(p.b_min, nb), math.ceil(np.float32(p.kappa_min) * np.float32(nb)))
        assert Bk.keep_budget(p.h_min, nb, p) == min(nb, low)
        assert Bk.keep_budget(0.0, nb, p) == min(nb, low)
        assert Bk.keep_budget(-3.0, nb, p) == min(nb, low)
    assert Bk.keep_budget(5.0, 0, p) == 0
    # nb below B_min keeps everything.
    assert Bk.keep_budget(0.0, 3, p) == 3


def test_budget_monotone_and_midpoint():
    p = _params()
    hs = np.linspace(0, 12, 2001)
    for nb in (37, 512, 8192):
        ks = [Bk.keep_budget(h, nb, p) for h in hs]
        assert all(a <= b for a, b in zip(ks, ks[1:]))
    # Midpoint of the entropy range keeps about kappa_min + (1-kappa_min)/2 of the blocks.
    mid = (p.h_min + p.log_v) / 2
    k = Bk.keep_budget(mid, 1000, p)
    assert abs(k - 1000 * (p.kappa_min + (1 - p.kappa_min) / 2)) <= 1


def test_budget_safety_margin_raises_budget():
    p0 = _params()
    p1 = _params(eps_h=0.5)
    for h in np.linspace(2.0, 11.0, 50):
        assert Bk.keep_budget(h, 700, p1) >= Bk.keep_budget(h, 700, p0)
    assert Bk.keep_budget(6.0, 700, p1) == Bk.keep_budget(6.5, 700, p0)


def test_select_blocks_brute_force_and_ties():
    kept, theta = Bk.select_blocks(np.array([1.0, 2.0, 2.0, 3.0]), 2)
    assert theta == 2.0 and list(kept) == [1, 2, 3]
    kept, theta = Bk.select_blocks(np.array([5.0, 1.0]), 0)
    assert len(kept) == 0 and theta == math.inf
    rng = np.random.default_rng(5)
    for trial in range(50):
        nb = int(rng.integers(1, 300))
        s = rng.integers(0, 40, nb).astype(float)   # many ties
        k = int(rng.integers(1, nb + 1))
        kept, theta = Bk.select_blocks(s, k)
        order = sorted(s, reverse=True)
        assert theta == order[k - 1]
        assert list(kept) == [b for b in range(nb) if s[b] >= theta]
        assert len(kept) >= k
