"""GPU-vs-oracle comparison of one decode step (used by the GPU tests and smoke()).

Per stage, the oracle is fed the GPU's own upstream values (teacher forcing):
its entropy for the block budget, its block summaries for the scores, its
kept list for attention, its temperature for sampling.  Bands:

* entropy (or its top-k / tail-corrected estimate), entropic time,
  temperature: |delta| <= 1e-4 (nats / absolute);
* kept list: bit-exact, except blocks whose oracle score lies within 1e-6
  of the oracle threshold; the GPU's list must also be exactly the blocks
  whose GPU score reaches the k-th largest GPU score, with k the budget the
  oracle computes (in float32) from the GPU's entropy;
* block scores: |delta| <= 1e-8 + 4e-6 |ref| (float32 arithmetic of each
  head's term; see SCORE_REL);
* attention output and log-sum-exp: |delta| <= 2e-3 + 2e-3 |ref|;
* token: equal, or, when the oracle's margin to a CDF edge is below 1e-6,
  a token whose CDF interval contains u within that margin.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Iterable, List, Optional

import numpy as np

from oracle import attention as OA
from oracle import blocks as OB
from oracle import entropy as OE
from oracle import layout as OL
from oracle import sample as OS

H_TOL = 1e-4
THETA_BAND = 1e-6
ATT_ABS = 2e-3
ATT_REL = 2e-3
TOKEN_BAND = 1e-6
# Block scores I_b: |delta| <= SCORE_ABS + SCORE_REL |I_b|.  Each head's
# term e^(l - L) (L - z) is formed in float32: the exponential's argument
# carries about |l - L| + 2 ulp of relative error and L - z about
# (|L| + |z|) ulp of its operands, so with |L|, |l - L| ~ 12 and |z| up to
# ~50 (large score ranges) the relative error stays below ~150 u = 9e-6 in
# the worst case and near 30 u = 2e-6 for ordinary rows; SCORE_ABS covers
# scores that underflow toward zero.
SCORE_ABS = 1e-8
SCORE_REL = 4e-6
# Largest errors seen in this process (reported at the end of a test run).
SEEN = {"score_rel": 0.0, "score_abs": 0.0, "att": 0.0, "h": 0.0}


@dataclass
class StepResult:
    """GPU outputs of one step, copied to host (numpy)."""
    h: np.ndarray
    tau: np.ndarray
    temp_next: np.ndarray
    temp_used: np.ndarray
    ksum: np.ndarray
    kept: np.ndarray
    n_kept: np.ndarray
    scores: np.ndarray
    theta: np.ndarray
    out: np.ndarray
    lse: np.ndarray
    tokens: np.ndarray
    kappa: Optional[np.ndarray] = None


@dataclass
class Report:
    failures: List[str] = field(default_factory=list)
    notes: List[str] = field(default_factory=list)
    band_exempt: int = 0
    max_att_err: float = 0.0
    max_h_err: float = 0.0
    max_score_err: float = 0.0
    max_score_rel_err: float = 0.0

    def fail(self, msg):
        self.failures.append(msg)

    def ok(self):
        return not self.failures


def collect(dev, with_kappa: bool = False) -> StepResult:
    c = lambda t: t.detach().cpu().numpy().copy()  # noqa: E731
    return StepResult(h=c(dev.h), tau=c(dev.tau), temp_next=c(dev.temp), temp_used=c(dev.temp_used),
                      ksum=c(dev.ksum), kept=c(dev.kept), n_kept=c(dev.n_kept), scores=c(dev.scores),
                      theta=c(dev.theta), out=c(dev.out), lse=c(dev.lse), tokens=c(dev.tokens),
                      kappa=c(dev.kappa) if with_kappa else None)


def check_step(*, k_pool, v_pool, tables, ctx_lens, q, logits, uniforms, h_prev, tau, temp,
               params, gpu: StepResult, block_size: int = 16, seqs: Optional[Iterable[int]] = None,
               check_ksum: bool = True, report: Optional[Report] = None, kappa=None) -> Report:
    """Compare the GPU step `gpu` with the oracle on sequences `seqs` (default all).

    The input arrays are the host copies of what the GPU step consumed
    (state before the step; `kappa`: the kept-fraction state, None when the
    step ran without it)."""
    rep = report or Report()
    B = len(ctx_lens)
    for s in (range(B) if seqs is None else seqs):
        N = int(ctx_lens[s])
        z = np.asarray(logits[s], dtype=np.float64)
        T = float(temp[s])
        # Stage 1: entropy (or the configured estimate of it) and controller.
        h_o = OE.control_entropy(z, T, params)
        dh = abs(float(gpu.h[s]) - h_o)
        rep.max_h_err = max(rep.max_h_err, dh)
        if dh > H_TOL:
            rep.fail(f"seq {s}: entropy {gpu.h[s]} vs oracle {h_o}")
        tau_o = OE.entropic_time(float(tau[s]), float(h_prev[s]), h_o)
        if abs(float(gpu.tau[s]) - tau_o) > H_TOL:
            rep.fail(f"seq {s}: tau {gpu.tau[s]} vs oracle {tau_o}")
        tn_o = OE.temperature_next(T, h_o, params.h_target, params.eta, params.t_min, params.t_max,
                                   params.rho_t)
        if abs(float(gpu.temp_next[s]) - tn_o) > H_TOL:
            rep.fail(f"seq {s}: next temperature {gpu.temp_next[s]} vs oracle {tn_o}")
        if float(gpu.temp_used[s]) != np.float32(T):
            rep.fail(f"seq {s}: temp_used {gpu.temp_used[s]} != input temperature {T}")

        # Stage 2: summaries, scores, budget and kept set.
        K, V = OL.gather_sequence(k_pool, v_pool, tables[s], N, block_size)
        counts = OB.block_token_counts(N, block_size)
        nb = len(counts)
        phys = np.asarray(tables[s][:nb], dtype=np.int64)
        kbar_g = gpu.ksum[phys].astype(np.float64) if nb else np.zeros((0,) + gpu.ksum.shape[1:])
        if check_ksum and nb:
            kbar_o = OB.block_means(K, block_size)
            err = np.abs(kbar_g - kbar_o)
            if np.any(err > 1e-5 + 1e-5 * np.abs(kbar_o)):
                rep.fail(f"seq {s}: block summaries differ by {err.max():.3g}")
        qs = OL.to_f64(q[s])
        kp = math.nan if kappa is None else float(kappa[s])
        k_o = OB.keep_budget(float(gpu.h[s]), nb, params, kp)
        if gpu.kappa is not None and nb:
            ka_o = OB.kept_fraction(float(gpu.h[s]), params, kp)
            if np.float32(gpu.kappa[s]) != ka_o:
                rep.fail(f"seq {s}: kept-fraction state {gpu.kappa[s]} vs oracle {ka_o}")
        nk = int(gpu.n_kept[s])
        kept_g = gpu.kept[s][:nk].astype(np.int64)
        if nb == 0:
            if nk != 0:
                rep.fail(f"seq {s}: empty sequence kept {nk} blocks")
        else:
            if getattr(params, "scoring", 0) == 1:
                I_o = OB.exact_token_scores(qs, K, block_size, params.scale)
            else:
                I_o, _, _ = OB.block_scores(qs, kbar_g, counts, params.scale)
            I_g = gpu.scores[s][:nb].astype(np.float32)
            serr = np.abs(I_g.astype(np.float64) - I_o)
            rep.max_score_err = max(rep.max_score_err, float(serr.max(initial=0.0)))
            big = np.abs(I_o) > SCORE_ABS / SCORE_REL
            if np.any(big):
                rep.max_score_rel_err = max(rep.max_score_rel_err,
                                            float((serr[big] / np.abs(I_o[big])).max()))
            if np.any(serr > SCORE_ABS + SCORE_REL * np.abs(I_o)):
                rep.fail(f"seq {s}: block scores differ by {serr.max():.3g}")
            forced = OB.forced_blocks(nb, getattr(params, "keep_first", 0),
                                      getattr(params, "keep_last", 0))
            _, theta_o = OB.select_blocks(I_o, k_o, forced)
            k_eff = max(k_o, len(forced))
            # GPU self-consistency, bit-exact on its own scores (forced blocks
            # rank above every score).
            rank_g = I_g.copy()
            rank_g[forced] = np.float32(np.inf)
            if k_eff > 0:
                theta_g_expect = np.sort(rank_g)[::-1][k_eff - 1]
                if np.float32(gpu.theta[s]) != theta_g_expect:
                    rep.fail(f"seq {s}: GPU threshold {gpu.theta[s]} is not the k={k_eff}-th "
                             f"largest GPU score {theta_g_expect}")
                expect = np.nonzero(rank_g >= np.float32(gpu.theta[s]))[0]
                if not np.array_equal(expect, kept_g):
                    rep.fail(f"seq {s}: GPU kept list is not its scores >= its threshold")
            elif nk != 0:
                rep.fail(f"seq {s}: budget 0 but {nk} blocks kept")
            # Oracle band.
            rank_o = I_o.copy()
            rank_o[forced] = np.inf
            with np.errstate(invalid="ignore"):
                must = set(np.nonzero(rank_o > theta_o + THETA_BAND)[0].tolist()) | \
                    set(forced.tolist())
                never = set(np.nonzero(rank_o < theta_o - THETA_BAND)[0].tolist())
                rep.band_exempt += int(np.sum(np.abs(rank_o - theta_o) <= THETA_BAND))
            kg = set(kept_g.tolist())
            if not must <= kg:
                rep.fail(f"seq {s}: {len(must - kg)} blocks above the threshold band not kept")
            if kg & never:
                rep.fail(f"seq {s}: {len(kg & never)} blocks below the threshold band kept")

        # Stage 3: attention over the GPU's kept blocks.
        o_ref, lse_ref = OA.sparse_decode(qs, K, V, kept_g, block_size, params.scale)
        o_g = gpu.out[s].astype(np.float64)
        err = np.abs(o_g - o_ref)
        rep.max_att_err = max(rep.max_att_err, float(err.max(initial=0.0)))
        if np.any(err > ATT_ABS + ATT_REL * np.abs(o_ref)):
            rep.fail(f"seq {s}: attention output differs by {err.max():.3g}")
        lg = gpu.lse[s].astype(np.float64)
        fin = np.isfinite(lse_ref)
        if not np.array_equal(fin, np.isfinite(lg)) or \
                np.any(np.abs(lg[fin] - lse_ref[fin]) > ATT_ABS + ATT_REL * np.abs(lse_ref[fin])):
            rep.fail(f"seq {s}: attention log-sum-exp differs")

        # Stage 4: sampling at the GPU's temperature.
        Tu = OE.effective_temperature(float(gpu.temp_used[s]), params)
        u = float(uniforms[s])
        x_o, margin = OS.sample(z, Tu, u)
        x_g = int(gpu.tokens[s])
        if x_g != x_o:
            ok = False
            if margin < TOKEN_BAND and 0 <= x_g < len(z):
                lo, hi = OS.cdf_interval(z, Tu, x_g)
                ok = (lo - TOKEN_BAND <= u < hi + TOKEN_BAND) and hi > lo
            if not ok:
                rep.fail(f"seq {s}: token {x_g} vs oracle {x_o} (margin {margin:.3g})")
            else:
                rep.notes.append(f"seq {s}: token {x_g} accepted in the tie band (oracle {x_o})")
    SEEN["score_rel"] = max(SEEN["score_rel"], rep.max_score_rel_err)
    SEEN["score_abs"] = max(SEEN["score_abs"], rep.max_score_err)
    SEEN["att"] = max(SEEN["att"], rep.max_att_err)
    SEEN["h"] = max(SEEN["h"], rep.max_h_err)
    return rep


def run_step(dec, dev, step: int = 0, stream=None, fused: bool = True, kappa: bool = False):
    """Issue one decode step of the uploaded inputs on the library (no sync):
    ent_decode_step when `fused`, else the four per-stage entry points; with
    `kappa` the kept-fraction state dev.kappa rides along."""
    B = dev.ctx_lens.shape[0]
    dec.step(B, logits=dev.logits[step], h_prev=dev.h_prev, tau=dev.tau, temp=dev.temp,
             q=dev.q[step], k_cache=dev.k_pool, v_cache=dev.v_pool, block_tables=dev.block_tables,
             ctx_lens=dev.ctx_lens, ksum=dev.ksum, uniforms=dev.uniforms[step], h=dev.h,
             temp_used=dev.temp_used, row_stats=dev.row_stats, kept=dev.kept, n_kept=dev.n_kept,
             out=dev.out, tokens=dev.tokens, lse=dev.lse, scores=dev.scores, theta=dev.theta,
             stream=stream, fused=fused, kappa=dev.kappa if kappa else None)
