"""Entropy-aware scheduling (oracle).  Test infrastructure: see the package
docstring.

Section 3.1 scores each active sequence s with

    pi(s) = E[Delta H_s] / (alpha C_s + beta M_s + gamma L_s)

and advances the best ones; Section 7 (stability of entropy-aware
scheduling) asks that every term be nonnegative and bounded and argues
that no sequence starves.  Readings (the paper gives symbols only):

* E[Delta H_s]: an exponentially weighted mean of the sequence's
  irreversible entropy drops Delta H+ (the increments of its entropic time
  tau), updated once per step the sequence ran: g <- (1 - lam) g + lam d,
  d = tau - tau_last.  It is floored at gain_floor > 0 so that no priority
  is zero.
* C_s: expected compute, the blocks the sequence kept at its last step.
* M_s: memory pressure, the blocks it holds, ceil(N_s / 16).
* L_s: latency risk, read as the sequence's remaining slack against a
  service-level objective of `slo` steps, max(slack_floor, slo - age_s),
  with age_s the steps since it last ran: the longer it waits, the smaller
  the slack and the higher its priority (the no-starvation argument needs
  priority to grow with waiting; a cost growing with waiting would do the
  opposite).
* The B_sel largest priorities are selected; equal priorities go to the
  lower index.  Selected sequences get age 0, the others age + 1.

Priorities decide an integer selection, so they are evaluated in float32 in
a fixed operation order, as the library does.
"""
from __future__ import annotations

import math

import numpy as np

f32 = np.float32


def update_gain(gain: float, tau: float, tau_last: float, ran: bool, lam: float):
    """EWMA of the entropy drop since the last call, for a sequence that ran
    (age 0) since then; others keep their mean.  Returns (gain, tau_last)."""
    if not ran:
        return f32(gain), f32(tau_last)
    d = f32(tau) - f32(tau_last)
    g = (f32(1.0) - f32(lam)) * f32(gain) + f32(lam) * d
    return f32(g), f32(tau)


def priority(gain: float, kept_blocks: int, ctx_len: int, age: int, prm) -> np.float32:
    """pi(s) in float32, in this operation order (no fused multiply-add)."""
    num = max(f32(gain), f32(prm.gain_floor))
    held = f32((max(int(ctx_len), 0) + 15) // 16)
    slack = max(f32(prm.slo) - f32(age), f32(prm.slack_floor))
    den = f32(prm.alpha) * f32(max(int(kept_blocks), 0))
    den = den + f32(prm.beta) * held
    den = den + f32(prm.gamma) * slack
    return f32(num / den)


def select(pri: np.ndarray, b_sel: int) -> np.ndarray:
    """Indices of the b_sel largest priorities (ties: lower index first),
    returned in ascending index order."""
    n = len(pri)
    kk = min(max(int(b_sel), 0), n)
    order = sorted(range(n), key=lambda i: (-float(pri[i]), i))
    return np.array(sorted(order[:kk]), dtype=np.int64)


def schedule(tau, tau_last, gain, age, n_kept, ctx_lens, b_sel, prm):
    """One scheduling call over the pool.  Returns the selected indices, the
    priorities and the updated state (tau_last, gain, age)."""
    n = len(tau)
    g = np.empty(n, dtype=np.float32)
    tl = np.empty(n, dtype=np.float32)
    pri = np.empty(n, dtype=np.float32)
    for s in range(n):
        g[s], tl[s] = update_gain(gain[s], tau[s], tau_last[s], int(age[s]) == 0, prm.ewma_rate)
        pri[s] = priority(g[s], int(n_kept[s]), int(ctx_lens[s]), int(age[s]), prm)
    sel = select(pri, b_sel)
    new_age = np.asarray(age, dtype=np.int64) + 1
    new_age[sel] = 0
    return sel, pri, tl, g, new_age.astype(np.int32)
