"""Decode attention restricted to the kept blocks (oracle, float64).

Test infrastructure: see the package docstring.
"""
from __future__ import annotations

import math

import numpy as np


def sparse_decode(q: np.ndarray, K: np.ndarray, V: np.ndarray, kept: np.ndarray,
                  block_size: int, scale: float):
    """Attention of one decode query over the tokens of the kept blocks only
    (Section 3.2: attention computation is restricted to the kept set).

    q [H_q, d]; K, V [N, H_kv, d] logical tokens; kept: logical block ids.
    For head h (KV head g = h // G), over valid tokens i of the kept blocks:
      s_i = scale <q_h, K_i,g>,  o_h = sum_i softmax(s)_i V_i,g,  lse_h = logsumexp_i s_i.
    Reading: the softmax is renormalised over the kept tokens; keeping every
    block gives dense decode attention.  An empty kept set gives o = 0 and
    lse = -inf.  Returns (o [H_q, d], lse [H_q])."""
    Hq, d = q.shape
    N, Hkv, _ = K.shape
    G = Hq // Hkv
    toks = [np.arange(b * block_size, min((b + 1) * block_size, N)) for b in kept]
    idx = np.concatenate(toks) if toks else np.zeros(0, dtype=np.int64)
    o = np.zeros((Hq, d))
    lse = np.full(Hq, -math.inf)
    if idx.size == 0:
        return o, lse
    for h in range(Hq):
        g = h // G
        s = float(scale) * (K[idx, g, :] @ q[h])
        m = s.max()
        w = np.exp(s - m)
        l = w.sum()
        o[h] = (w @ V[idx, g, :]) / l
        lse[h] = m + math.log(l)
    return o, lse
