"""Pins of the exact token-level scoring mode and the forced keeps (oracle).

Exact scores (Section 3.2 with a_i the softmax of the current query over
every valid key): a brute force from library routines (scipy's softmax and
elementwise -x log x) summed per block; the sum over blocks equals the mean
attention entropy (scipy.stats.entropy); q = 0 gives (n_b / N) log N;
permuting tokens inside a block changes nothing.  Forced keeps: the forced
set on short and long sequences; the kept set against a sort-based brute
force (forced blocks always kept and counted in the budget, the rest the
top scores with ties).
"""
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats

from oracle import blocks as Bk


def _brute(q, K, bs, scale):
    Hq = q.shape[0]
    N, Hkv, _ = K.shape
    G = Hq // Hkv
    nb = -(-N // bs)
    out = np.zeros(nb)
    for h in range(Hq):
        w = scipy.special.softmax(scale * (K[:, h // G, :] @ q[h]))
        c = scipy.special.entr(w)
        for i in range(N):
            out[i // bs] += c[i]
    return out / Hq


@pytest.mark.parametrize("N,Hq,Hkv", [(1, 2, 1), (16, 4, 2), (53, 4, 2), (200, 8, 2), (97, 6, 3)])
def test_exact_scores_brute_force_and_entropy_sum(N, Hq, Hkv):
    rng = np.random.default_rng(N + Hq)
    d, bs, scale = 8, 16, 0.4
    K = rng.normal(size=(N, Hkv, d)) * 1.5
    q = rng.normal(size=(Hq, d))
    I = Bk.exact_token_scores(q, K, bs, scale)
    assert I.shape == (-(-N // bs),)
    assert np.allclose(I, _brute(q, K, bs, scale), rtol=1e-12, atol=1e-14)
    G = Hq // Hkv
    Hmean = np.mean([scipy.stats.entropy(scipy.special.softmax(scale * (K[:, h // G] @ q[h])))
                     for h in range(Hq)])
    assert abs(I.sum() - Hmean) < 1e-12
    assert np.all(I >= 0)


def test_exact_scores_uniform_attention():
    N, bs = 75, 16
    K = np.random.default_rng(1).normal(size=(N, 2, 8))
    I = Bk.exact_token_scores(np.zeros((4, 8)), K, bs, 0.3)
    n = Bk.block_token_counts(N, bs)
    assert np.allclose(I, n / N * math.log(N), rtol=1e-13)


def test_exact_scores_permutation_inside_blocks():
    rng = np.random.default_rng(2)
    N, bs = 70, 16
    K = rng.normal(size=(N, 2, 8))
    q = rng.normal(size=(4, 8))
    I = Bk.exact_token_scores(q, K, bs, 0.5)
    P = K.copy()
    for b0 in range(0, N, bs):
        idx = np.arange(b0, min(b0 + bs, N))
        P[idx] = K[rng.permutation(idx)]
    assert np.allclose(Bk.exact_token_scores(q, P, bs, 0.5), I, rtol=1e-12, atol=1e-15)
    # Swapping two tokens across blocks moves exactly their contributions.
    S = K.copy()
    S[[3, 40]] = K[[40, 3]]
    Is = Bk.exact_token_scores(q, S, bs, 0.5)
    assert abs(Is.sum() - I.sum()) < 1e-12
    assert np.allclose(Is[1], I[1]) and not np.isclose(Is[0], I[0])


def test_forced_blocks():
    assert Bk.forced_blocks(5, 1, 1).tolist() == [0, 4]
    assert Bk.forced_blocks(1, 1, 1).tolist() == [0]
    assert Bk.forced_blocks(3, 2, 2).tolist() == [0, 1, 2]
    assert Bk.forced_blocks(10, 0, 0).tolist() == []
    assert Bk.forced_blocks(10, 0, 3).tolist() == [7, 8, 9]
    assert Bk.forced_blocks(0, 2, 2).tolist() == []


@pytest.mark.parametrize("seed", range(6))
def test_forced_selection_brute_force(seed):
    rng = np.random.default_rng(seed)
    nb = int(rng.integers(1, 40))
    scores = rng.choice(rng.random(6), size=nb) if seed % 2 else rng.random(nb)
    for kf, kl in ((1, 1), (0, 2), (3, 0), (2, 5)):
        F = Bk.forced_blocks(nb, kf, kl)
        for k in range(0, nb + 1):
            kept, theta = Bk.select_blocks(scores, k, F)
            assert set(F.tolist()) <= set(kept.tolist())
            assert list(kept) == sorted(kept)
            rest = [b for b in range(nb) if b not in set(F.tolist())]
            m = max(k, len(F)) - len(F)
            if m == 0:
                assert kept.tolist() == F.tolist() and theta == math.inf
                continue
            srt = sorted((scores[b] for b in rest), reverse=True)
            th = srt[m - 1]
            assert theta == th
            assert sorted(set(kept.tolist()) - set(F.tolist())) == [b for b in rest if scores[b] >= th]
    # No forced blocks: the unforced selection.
    k2, t2 = Bk.select_blocks(scores, 3, np.zeros(0, dtype=np.int64))
    k1, t1 = Bk.select_blocks(scores, 3)
    assert k1.tolist() == k2.tolist() and t1 == t2
