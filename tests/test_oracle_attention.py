"""Pins of the oracle's kept-block decode attention.

Keep-all must equal dense attention (explicit loops, and torch's CPU
scaled_dot_product_attention in float64 as a library cross-check); one kept
block must equal attention over only its tokens; closed forms for a zero
query and identical value rows.
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as A


def _dense_loops(q, K, V, toks, scale):
    Hq, d = q.shape
    G = Hq // K.shape[1]
    o = np.zeros((Hq, d))
    lse = np.zeros(Hq)
    for h in range(Hq):
        s = [scale * sum(q[h, j] * K[i, h // G, j] for j in range(d)) for i in toks]
        m = max(s)
        w = [math.exp(x - m) for x in s]
        tot = sum(w)
        for i, wi in zip(toks, w):
            o[h] += wi / tot * V[i, h // G]
        lse[h] = m + math.log(tot)
    return o, lse


@pytest.mark.parametrize("N,G", [(1, 1), (16, 2), (37, 4), (50, 1)])
def test_keep_all_equals_dense_loops(N, G):
    rng = np.random.default_rng(N)
    Hkv, d = 2, 8
    q = rng.normal(size=(Hkv * G, d))
    K = rng.normal(size=(N, Hkv, d))
    V = rng.normal(size=(N, Hkv, d))
    nb = -(-N // 16)
    o, lse = A.sparse_decode(q, K, V, np.arange(nb), 16, 0.35)
    ro, rl = _dense_loops(q, K, V, list(range(N)), 0.35)
    assert np.allclose(o, ro, rtol=1e-12, atol=1e-13)
    assert np.allclose(lse, rl, rtol=1e-12, atol=1e-13)


def test_keep_all_equals_torch_sdpa():
    rng = np.random.default_rng(9)
    Hkv, G, d, N = 4, 4, 64, 301
    q = rng.normal(size=(Hkv * G, d))
    K = rng.normal(size=(N, Hkv, d))
    V = rng.normal(size=(N, Hkv, d))
    o, _ = A.sparse_decode(q, K, V, np.arange(-(-N // 16)), 16, 1 / math.sqrt(d))
    qt = torch.from_numpy(q).reshape(1, Hkv * G, 1, d)
    kt = torch.from_numpy(np.repeat(K, G, axis=1).transpose(1, 0, 2).copy()).unsqueeze(0)
    vt = torch.from_numpy(np.repeat(V, G, axis=1).transpose(1, 0, 2).copy()).unsqueeze(0)
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=1 / math.sqrt(d))
    assert np.allclose(o, ref[0, :, 0].numpy(), rtol=1e-11, atol=1e-12)


def test_subset_equals_attention_over_its_tokens_only():
    rng = np.random.default_rng(2)
    Hkv, G, d, N = 2, 2, 8, 70
    q = rng.normal(size=(Hkv * G, d))
    K = rng.normal(size=(N, Hkv, d))
    V = rng.normal(size=(N, Hkv, d))
    o, lse = A.sparse_decode(q, K, V, np.array([1]), 16, 0.5)
    ro, rl = _dense_loops(q, K, V, list(range(16, 32)), 0.5)
    assert np.allclose(o, ro, rtol=1e-12) and np.allclose(lse, rl, rtol=1e-12)
    # partial last block: only its valid tokens
    o, lse = A.sparse_decode(q, K, V, np.array([0, 4]), 16, 0.5)
    ro, rl = _dense_loops(q, K, V, list(range(0, 16)) + list(range(64, 70)), 0.5)
    assert np.allclose(o, ro, rtol=1e-12) and np.allclose(lse, rl, rtol=1e-12)


def test_zero_query_and_identical_values():
    rng = np.random.default_rng(3)
    N, Hkv, d = 45, 2, 6
    K = rng.normal(size=(N, Hkv, d))
    V = rng.normal(size=(N, Hkv, d))
    kept = np.array([0, 2])
    o, lse = A.sparse_decode(np.zeros((2, d)), K, V, kept, 16, 0.3)
    toks = list(range(16)) + list(range(32, 45))
    assert np.allclose(o, V[toks].mean(axis=0), rtol=1e-12)
    assert np.allclose(lse, math.log(len(toks)), rtol=1e-14)
    row = rng.normal(size=(Hkv, d))
    V2 = np.broadcast_to(row, (N, Hkv, d)).copy()
    o, _ = A.sparse_decode(rng.normal(size=(4, d)), K, V2, kept, 16, 0.3)
    assert np.allclose(o, np.repeat(row, 2, axis=0), rtol=1e-12)


def test_empty_kept_set():
    o, lse = A.sparse_decode(np.ones((2, 4)), np.ones((3, 1, 4)), np.ones((3, 1, 4)),
                             np.zeros(0, dtype=np.int64), 16, 1.0)
    assert np.all(o == 0) and np.all(lse == -np.inf)
