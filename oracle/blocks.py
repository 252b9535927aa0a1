"""Block summaries, block entropic contributions and the kept-block set (oracle, float64).

Test infrastructure: see the package docstring.

The paper defines a block's entropic contribution as the attention-weighted
surprisal of its tokens and keeps the blocks whose contribution reaches a
threshold set by the entropy regime (Section 3.2), with a safety floor and a
minimum block budget (Section 3.3, "Conservative pruning under uncertainty
bounds"; Section 5, "Robust control with uncertainty floors").  It does not
say how the attention weights are obtained before attention runs, what the
surprisal's distribution is, or what form the threshold takes.  Readings:

* weights: the current query's softmax over tokens when every token carries
  its block's mean key (one mean key per block and KV head);
* surprisal: -log of that same weight, so a block's score is its additive
  share of the attention entropy;
* heads: one score per block, the mean over all query heads;
* threshold: the k-th largest score, with the budget k growing linearly in
  the (floored) entropy from kappa_min * nb at H_min to nb at log |V|;
  ties at the threshold are all kept.

The exact token-level weights (every key of the sequence against the current
query) are the second scoring mode, exact_token_scores.  Optionally the first
and last blocks of a sequence are always kept (forced_blocks).

These readings are the build's; the paper prints no values to pin them to
(parity unpinned against the paper; pinned here against closed forms of the
readings themselves).
"""
from __future__ import annotations

import math

import numpy as np


def block_token_counts(n_tokens: int, block_size: int) -> np.ndarray:
    """Valid tokens per logical block: block_size, except a partial last block."""
    nb = -(-n_tokens // block_size)
    n = np.full(nb, block_size, dtype=np.int64)
    if nb:
        n[-1] = n_tokens - block_size * (nb - 1)
    return n


def block_means(K: np.ndarray, block_size: int) -> np.ndarray:
    """Mean key of each block over its valid tokens: K [N, H_kv, d] -> [nb, H_kv, d]."""
    N = K.shape[0]
    counts = block_token_counts(N, block_size)
    out = np.empty((len(counts),) + K.shape[1:])
    for b, n in enumerate(counts):
        out[b] = K[b * block_size: b * block_size + n].sum(axis=0) / n
    return out


def block_scores(q: np.ndarray, kbar: np.ndarray, counts: np.ndarray, scale: float):
    """Block entropic contributions I_b (Section 3.2) under the mean-key reading.

    For query head h with KV head g = h // G:
      z_bh  = scale <q_h, kbar_bg>             logit every token of block b gets
      a_bh  = exp(z_bh) / sum_b' n_b' exp(z_b'h)   weight of one token of b
      I_bh  = n_b * a_bh * (-log a_bh)           sum over the block's tokens
    and I_b = mean_h I_bh.  Returns (I [nb], I_per_head [nb, H_q], z [nb, H_q])."""
    Hq, d = q.shape
    nb, Hkv, _ = kbar.shape
    G = Hq // Hkv
    z = np.empty((nb, Hq))
    for h in range(Hq):
        z[:, h] = float(scale) * (kbar[:, h // G, :] @ q[h])
    I_h = np.empty((nb, Hq))
    for h in range(Hq):
        # log of the normaliser sum_b n_b exp(z_b), written as a log-sum-exp.
        ell = z[:, h] + np.log(counts)
        m = ell.max()
        L = m + math.log(np.sum(np.exp(ell - m)))
        log_a = z[:, h] - L                      # log weight of one token of block b
        I_h[:, h] = counts * np.exp(log_a) * (-log_a)
    return I_h.mean(axis=1), I_h, z


def kept_fraction(h: float, params, kappa_prev: float = math.nan) -> np.float32:
    """Kept fraction kappa from the entropy H_t (reading of the
    entropy-driven threshold and its guards; Sections 3.2, 3.3, 5):

      H_g   = max(H + eps_H, H_min)                  conservative, floored entropy
      u     = clip((H_g - H_min) / (log|V| - H_min), 0, 1)
      kappa = kappa_min + (1 - kappa_min) u

    and the bounded rate of change of Section 5 (guard iii), read as a bound
    on how fast pruning may tighten: kappa >= kappa_prev - dkappa when the
    previous step's fraction is known (NaN: no previous step); a larger
    fraction is always allowed.

    Evaluated in float32 with exactly this operation order (no fused
    multiply-add): the block count is an integer decided by floating point,
    and both sides must take that decision in the same precision."""
    f = np.float32
    hg = max(f(h) + f(params.eps_h), f(params.h_min))
    u = (hg - f(params.h_min)) / (f(params.log_v) - f(params.h_min))
    u = min(max(u, f(0.0)), f(1.0))
    kappa = f(params.kappa_min) + (f(1.0) - f(params.kappa_min)) * u
    if not math.isnan(kappa_prev):
        kappa = max(kappa, f(kappa_prev) - f(getattr(params, "dkappa", 1.0)))
    return f(kappa)


def keep_budget(h: float, nb: int, params, kappa_prev: float = math.nan) -> int:
    """Number of blocks to keep, k = min(nb, max(min(B_min, nb), ceil(kappa nb)))
    with kappa = kept_fraction(h, params, kappa_prev) (float32)."""
    if nb <= 0:
        return 0
    f = np.float32
    kappa = kept_fraction(h, params, kappa_prev)
    k = int(np.ceil(f(kappa * f(nb))))
    return min(nb, max(min(int(params.b_min), nb), k))


def forced_blocks(nb: int, keep_first: int = 0, keep_last: int = 0) -> np.ndarray:
    """Blocks always kept: the first keep_first and the last keep_last logical
    blocks of a sequence of nb blocks (a build option; the paper prunes by
    score alone)."""
    f = set(range(min(max(int(keep_first), 0), nb)))
    f |= set(range(max(nb - max(int(keep_last), 0), 0), nb))
    return np.array(sorted(f), dtype=np.int64)


def select_blocks(scores: np.ndarray, k: int, forced=None):
    """Kept set B_t = {b : I_b >= theta_t} with theta_t the k-th largest score
    (Section 3.2), listed in ascending block order.  Ties at theta are kept.
    Returns (kept indices, theta); theta is +inf when k == 0.

    Forced blocks (optional) are always kept and count toward the budget:
    they rank above every score, the budget becomes max(k, |forced|), and
    theta is the budget-th largest of those ranks (+inf when the forced
    blocks fill it)."""
    nb = len(scores)
    nf = 0 if forced is None else len(forced)
    if nf:
        ranked = np.asarray(scores, dtype=np.float64).copy()
        ranked[np.asarray(forced, dtype=np.int64)] = math.inf
        k = max(int(k), nf)
    else:
        ranked = scores
    if k <= 0 or nb == 0:
        return np.zeros(0, dtype=np.int64), math.inf
    theta = float(np.sort(ranked)[::-1][k - 1])
    kept = np.nonzero(ranked >= theta)[0]
    return kept.astype(np.int64), theta


def exact_token_scores(q: np.ndarray, K: np.ndarray, block_size: int, scale: float) -> np.ndarray:
    """Block entropic contributions from the exact token-level attention
    weights (Section 3.2 taken literally: a_i is the current query's softmax
    over all valid keys, surprisal -log a_i), I_b = mean_h sum_{i in b}
    a_i (-log a_i).  The conservative scoring mode: it reads every key of the
    sequence, where the mean-key reading reads one summary per block."""
    Hq, d = q.shape
    N, Hkv, _ = K.shape
    G = Hq // Hkv
    nb = -(-N // block_size)
    out = np.zeros(nb)
    for h in range(Hq):
        s = float(scale) * (K[:, h // G, :] @ q[h])
        m = s.max()
        log_a = s - (m + math.log(np.sum(np.exp(s - m))))
        contrib = np.exp(log_a) * (-log_a)
        for b in range(nb):
            out[b] += contrib[b * block_size:(b + 1) * block_size].sum()
    return out / Hq
