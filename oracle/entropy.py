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


def _topk_split(z: np.ndarray, temp: float, k: int):
    """The k largest log-probabilities of the tempered softmax (the top-k set
    K_t of Section 2.1) and the rest.  With ties at the k-th value any choice
    of members gives the same multiset of probabilities, so everything below
    is well defined.  k is clamped to [1, |V|]."""
    logp = tempered_log_softmax(z, temp)
    kk = min(max(int(k), 1), logp.size)
    desc = np.sort(logp)[::-1]
    return desc[:kk], desc[kk:], kk


def topk_entropy(z: np.ndarray, temp: float, k: int):
    """Top-k truncated entropy (Section 2.1, top-k approximation).

    K = the k most probable tokens under p; m = sum_{x in K} p(x);
    p~(x) = p(x) / m on K and 0 elsewhere; H~ = -sum_{x in K} p~(x) ln p~(x).
    Returns (H~, m, mbar) with mbar = 1 - m summed directly over the tokens
    outside K (more accurate than 1 - m when the tail is small)."""
    top, rest, _ = _topk_split(z, temp, k)
    p = np.exp(top)
    m = float(np.sum(p))
    mbar = float(np.sum(np.exp(rest))) if rest.size else 0.0
    pos = p > 0.0
    log_pt = top[pos] - math.log(m)           # log p~ on K
    h_tilde = float(-np.sum(np.exp(log_pt) * log_pt))
    return h_tilde, m, mbar


def binary_entropy(x: float) -> float:
    """h(x) = -x ln x - (1 - x) ln(1 - x), with h(0) = h(1) = 0."""
    x = float(x)
    if x <= 0.0 or x >= 1.0:
        return 0.0
    return -x * math.log(x) - (1.0 - x) * math.log1p(-x)


def tail_corrected_entropy(z: np.ndarray, temp: float, k: int) -> float:
    """Tail-corrected estimate (Section 2.1, tail-corrected estimator):

      H^ = H~ + h(mbar) + mbar ln(|V| - k)

    the bound on H obtained by taking the mass outside the top-k set as
    uniform over the |V| - k remaining tokens.  With k >= |V| there is no tail
    and the last term is 0 (0 ln 0 = 0)."""
    h_tilde, _, mbar = topk_entropy(z, temp, k)
    V = np.asarray(z).size
    kk = min(max(int(k), 1), V)
    tail = mbar * math.log(V - kk) if V > kk else 0.0
    return h_tilde + binary_entropy(mbar) + tail


# Estimator codes (the same values as the library configuration field).
EXACT, TOPK, TAIL = 0, 1, 2


def entropy_estimate(z: np.ndarray, temp: float, estimator: int = EXACT, k: int = 0) -> float:
    """The entropy the controller acts on (Section 3.3, estimator in the
    control loop): the exact H_t, the top-k H~_t, or the tail-corrected
    H^_t."""
    if estimator == EXACT:
        return entropy(z, temp)
    if estimator == TOPK:
        return topk_entropy(z, temp, k)[0]
    if estimator == TAIL:
        return tail_corrected_entropy(z, temp, k)
    raise ValueError(f"unknown estimator {estimator}")


def effective_temperature(temp: float, params) -> float:
    """Temperature of every softmax over the vocabulary in a step: the
    controlled T_t times the calibration temperature T_cal (Section 5,
    calibration-aware entropy, read as a post-hoc wrapper on the logits,
    p^cal proportional to exp(z / T_cal), to which the sampling temperature
    then applies; T_cal = 1 leaves the step unchanged)."""
    return float(temp) * float(getattr(params, "t_cal", 1.0))


def control_entropy(z: np.ndarray, temp: float, params) -> float:
    """The entropy the controller and the block budget act on: the
    configured estimate (exact, top-k or tail-corrected) of the entropy at
    the effective temperature, plus the injected bias of the miscalibration
    stress tests (Section 5, "injecting entropy bias"; 0 by default)."""
    h = entropy_estimate(z, effective_temperature(temp, params),
                         int(getattr(params, "estimator", EXACT)), int(getattr(params, "est_k", 0)))
    return h + float(getattr(params, "h_bias", 0.0))


def entropic_time(tau: float, h_prev: float, h: float) -> float:
    """tau + max(0, H_{t-1} - H_t)  (Section 2: entropy flow Delta H_t, its
    positive part, and entropic time as their running sum).

    Reading: a NaN previous entropy means "no previous step" and adds 0."""
    if math.isnan(h_prev):
        return float(tau)
    return float(tau) + max(0.0, float(h_prev) - float(h))


def temperature_next(temp: float, h: float, h_target: float, eta: float,
                     t_min: float, t_max: float, rho_t: float = math.inf) -> float:
    """T_{t+1} = clip(T_t exp(eta (H_t - H*)), T_min, T_max)  (Section 3.3).

    Reading: `eta` is a signed gain.  With the positive gain as printed the
    loop feeds back positively, because dH/dT >= 0 for a softmax; the
    stabilising law the paper describes (high entropy driven toward
    commitment) and its linearisation in Section 7 need eta < 0 here.

    Bounded rate of change (Section 5, guard iii): the multiplicative step
    exp(eta (H - H*)) is clipped to [exp(-rho_t), exp(rho_t)] before the
    clip to [T_min, T_max], so |ln T_{t+1} - ln T_t| <= rho_t inside the
    bounds; rho_t = inf leaves the law unchanged."""
    step = math.exp(float(eta) * (float(h) - float(h_target)))
    if math.isfinite(float(rho_t)):
        step = min(max(step, math.exp(-float(rho_t))), math.exp(float(rho_t)))
    t = float(temp) * step
    return min(max(t, float(t_min)), float(t_max))


def control_step(logits: np.ndarray, h_prev: np.ndarray, tau: np.ndarray, temp: np.ndarray,
                 params) -> dict:
    """One controller update for a batch of logit rows [B, V].

    H_t is measured at the current temperature T_t; sampling uses the same
    T_t; the updated temperature applies to the next step.  The controller
    acts on the configured estimate (exact by default; `params.estimator`,
    `params.est_k`).  Returns H_t, the updated tau, the temperature used and
    the next temperature."""
    B = logits.shape[0]
    h = np.empty(B)
    tau_out = np.empty(B)
    t_next = np.empty(B)
    for b in range(B):
        h[b] = control_entropy(logits[b], float(temp[b]), params)
        tau_out[b] = entropic_time(float(tau[b]), float(h_prev[b]), h[b])
        t_next[b] = temperature_next(float(temp[b]), h[b], params.h_target, params.eta,
                                     params.t_min, params.t_max,
                                     float(getattr(params, "rho_t", math.inf)))
    return {"h": h, "tau": tau_out, "temp_used": np.asarray(temp, dtype=np.float64).copy(),
            "temp_next": t_next}
