"""One whole entropic-time decode step for a batch (oracle, float64).

Test infrastructure: see the package docstring.

Per sequence, in the order of the closed loop of Section 3.4: entropy of the
next-token distribution at the current temperature, entropic time and the
temperature update; block scores and the kept set under the entropy-driven
budget; attention over the kept blocks; sampling at the current temperature.

Teacher forcing: a per-stage parity check feeds a stage the GPU's own
upstream values (its entropy, its block summaries), so that a discrete
decision downstream is compared on identical inputs.  The optional
``*_override`` arguments carry those values; without them the oracle runs
free from the raw inputs alone.
"""
from __future__ import annotations

import math
from typing import Iterable, Optional

import numpy as np

from . import attention, blocks, entropy, layout, sample


def sequence_step(s: int, *, k_pool, v_pool, tables, ctx_lens, q, logits, h_prev, tau, temp,
                  uniforms, params, block_size: int, h_override: Optional[float] = None,
                  ksum_pool: Optional[np.ndarray] = None, want_exact: bool = False,
                  kappa=None) -> dict:
    """Every output of the step for sequence s.  Array arguments are the
    batch's buffers in the library's layouts (one step's q/logits/uniforms);
    `kappa` holds the previous step's kept fractions (None or NaN: none)."""
    N = int(ctx_lens[s])
    z = np.asarray(logits[s], dtype=np.float64)
    T = float(temp[s])
    h = entropy.control_entropy(z, T, params)
    out = {
        "h": h,
        "tau": entropy.entropic_time(float(tau[s]), float(h_prev[s]), h),
        "temp_used": T,
        "temp_next": entropy.temperature_next(T, h, params.h_target, params.eta,
                                              params.t_min, params.t_max,
                                              float(getattr(params, "rho_t", math.inf))),
    }
    K, V = layout.gather_sequence(k_pool, v_pool, tables[s], N, block_size)
    qs = layout.to_f64(q[s])
    counts = blocks.block_token_counts(N, block_size)
    nb = len(counts)
    if ksum_pool is not None:
        kbar = np.asarray(ksum_pool[np.asarray(tables[s][:nb], dtype=np.int64)], dtype=np.float64)
    else:
        kbar = blocks.block_means(K, block_size)
    out["kbar"] = kbar
    if nb and getattr(params, "scoring", 0) == 1:
        I = blocks.exact_token_scores(qs, K, block_size, params.scale)
    elif nb:
        I, _, _ = blocks.block_scores(qs, kbar, counts, params.scale)
    else:
        I = np.zeros(0)
    h_budget = h if h_override is None else float(h_override)
    kp = math.nan if kappa is None else float(kappa[s])
    k = blocks.keep_budget(h_budget, nb, params, kp)
    out["kappa"] = float(blocks.kept_fraction(h_budget, params, kp)) if nb else kp
    forced = blocks.forced_blocks(nb, getattr(params, "keep_first", 0),
                                  getattr(params, "keep_last", 0))
    kept, theta = blocks.select_blocks(I, k, forced)
    out.update(scores=I, k=k, kept=kept, theta=theta, nb=nb)
    o, lse = attention.sparse_decode(qs, K, V, kept, block_size, params.scale)
    out.update(o=o, lse=lse)
    tok, margin = sample.sample(z, entropy.effective_temperature(T, params), float(uniforms[s]))
    out.update(token=tok, margin=margin)
    if want_exact and nb:
        out["exact_scores"] = blocks.exact_token_scores(qs, K, block_size, params.scale)
    return out


def decode_step(seqs: Optional[Iterable[int]] = None, **kw) -> list:
    """`sequence_step` for each sequence in `seqs` (default: the whole batch)."""
    B = len(kw["ctx_lens"])
    h_over = kw.pop("h_override", None)
    return [sequence_step(s, h_override=None if h_over is None else h_over[s], **kw)
            for s in (range(B) if seqs is None else seqs)]
