"""Entropy, entropic time and the temperature law (oracle, float64).

Test infrastructure: see the package docstring.
"""
from __future__ import annotations

import math

import numpy as np


def tempered_log_softmax(z: np.ndarray, temp: float) -> np.ndarray:
    """log p(x) for p(x) = exp(z(x)/T) / sum_y exp(z(y)/T)  (Section 2.1, exact-entropy display).

    Logits of -inf get log p = -inf (probability zero)."""
    y = np.asarray(z, dtype=np.float64) / float(temp)
    m = np.max(y)
    lse = m + math.log(np.sum(np.exp(y - m)))
    return y - lse


def entropy(z: np.ndarray, temp: float) -> float:
    """Exact Shannon entropy H = -sum_x p(x) log p(x) in nats over the full
    vocabulary, with p the tempered softmax (Section 2, definition of H_t;
    Section 2.1, exact entropy).

    Reading: natural logarithm; terms with p(x) = 0 contribute 0 (0 log 0 = 0);
    the row must hold at least one finite logit."""
    logp = tempered_log_softmax(z, temp)
    p = np.exp(logp)
    pos = p > 0.0
    return float(-np.sum(p[pos] * logp[pos]))


def entropic_time(tau: float, h_prev: float, h: float) -> float:
    """tau + max(0, H_{t-1} - H_t)  (Section 2: entropy flow Delta H_t, its
    positive part, and entropic time as their running sum).

    Reading: a NaN previous entropy means "no previous step" and adds 0."""
    if math.isnan(h_prev):
        return float(tau)
    return float(tau) + max(0.0, float(h_prev) - float(h))


def temperature_next(temp: float, h: float, h_target: float, eta: float,
                     t_min: float, t_max: float) -> float:
    """T_{t+1} = clip(T_t exp(eta (H_t - H*)), T_min, T_max)  (Section 3.3).

    Reading: `eta` is a signed gain.  With the positive gain as printed the
    loop feeds back positively, because dH/dT >= 0 for a softmax; the
    stabilising law the paper describes (high entropy driven toward
    commitment) and its linearisation in Section 7 need eta < 0 here."""
    t = float(temp) * math.exp(float(eta) * (float(h) - float(h_target)))
    return min(max(t, float(t_min)), float(t_max))


def control_step(logits: np.ndarray, h_prev: np.ndarray, tau: np.ndarray, temp: np.ndarray,
                 params) -> dict:
    """One controller update for a batch of logit rows [B, V].

    H_t is measured at the current temperature T_t; sampling uses the same
    T_t; the updated temperature applies to the next step.  Returns H_t,
    the updated tau, the temperature used and the next temperature."""
    B = logits.shape[0]
    h = np.empty(B)
    tau_out = np.empty(B)
    t_next = np.empty(B)
    for b in range(B):
        h[b] = entropy(logits[b], float(temp[b]))
        tau_out[b] = entropic_time(float(tau[b]), float(h_prev[b]), h[b])
        t_next[b] = temperature_next(float(temp[b]), h[b], params.h_target, params.eta,
                                     params.t_min, params.t_max)
    return {"h": h, "tau": tau_out, "temp_used": np.asarray(temp, dtype=np.float64).copy(),
            "temp_next": t_next}
