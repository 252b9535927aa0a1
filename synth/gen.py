"""Seeded synthetic inputs of a decode step, in the library's buffer layouts.

Recipe (all draws from NumPy PCG64):

* Root seed ``SEED_BASE + workload.index`` (or an explicit seed).  The root
  SeedSequence spawns one child for batch-level draws and one per sequence,
  so any sequence's data is reproducible on its own.
* Batch-level stream, in this order: context lengths; per-sequence logit
  scale s; previous-step entropy H_prev ~ U[0, log V]; sampling uniforms
  u ~ U[0,1) float32 for every step; the permutation that places logical
  blocks in the shared pool; the per-step drift of s (closed loop).
* Per-sequence stream, in this order: queries for every step; K tiles; V
  tiles; the planted key run; logits for every step; appended K/V tokens.
* bf16 values (keys, values, queries) are N(0,1) drawn by inverse-CDF
  sampling from a 16-bit uniform (a table of 65536 normal quantiles) and
  rounded to bf16 with round-to-nearest-even.  fp32 values are
  ``standard_normal`` in float32.
* Logits: N(0, s^2) with s ~ U[lo, hi] per sequence; or, for the skewed
  batch, even rows Zipf-peaked z_j = -1.2 log r_j (r a random permutation of
  the ranks 1..V, so the top token sits at a random index) and odd rows flat
  N(0, 0.3^2).  Closed loop: s follows a walk with N(0, 0.25^2) steps,
  reflected into [lo, hi].
* Planted run (long context): 64 consecutive tokens at a random offset whose
  key for KV head g is sqrt(d) (c u_g + sqrt(1-c^2) w) with c = 0.9, u_g the
  unit mean of group g's queries (step 0) and w a random unit vector
  orthogonal to u_g, drawn per token.

Layouts (the library's): K pool [P, H_kv, 16, d]; V pool [P, H_kv, d, 16]
(each (block, head) tile contiguous, V tile dim-major); block tables
[B, MAXB] int32 of physical block ids, -1 where unused; queries
[B, H_q, d]; logits [B, V] float32.

This module contains no arithmetic of the method itself.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional

import numpy as np

from .workloads import SEED_BASE, ZIPF_EXPONENT, Workload

_QUANTILE_BITS = None


def _normal_bf16_table() -> np.ndarray:
    global _QUANTILE_BITS
    if _QUANTILE_BITS is None:
        from scipy.special import ndtri
        q = ndtri((np.arange(65536, dtype=np.float64) + 0.5) / 65536.0).astype(np.float32)
        _QUANTILE_BITS = f32_to_bf16_bits(q)
    return _QUANTILE_BITS


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round to nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = u >> 16
    r &= 1
    r += 0x7FFF
    r += u
    r >>= 16
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def _normal_values(rng: np.random.Generator, shape, dtype: str) -> np.ndarray:
    """N(0,1) values: uint16 bf16 bits for "bf16", float32 for "f32"."""
    if dtype == "bf16":
        idx = rng.integers(0, 65536, size=shape, dtype=np.uint16)
        return _normal_bf16_table()[idx]
    return rng.standard_normal(size=shape, dtype=np.float32)


@dataclass
class Inputs:
    workload: Workload
    ctx_lens: np.ndarray        # int32 [B]      tokens in the cache at step 0
    block_tables: np.ndarray    # int32 [B, MAXB]
    num_pool_blocks: int
    k_pool: np.ndarray          # [P, Hkv, 16, d]   uint16 bf16 bits or float32
    v_pool: np.ndarray          # [P, Hkv, d, 16]
    q: np.ndarray               # [S, B, Hq, d]     one query per step
    logits: np.ndarray          # float32 [S, B, V]
    h_prev: np.ndarray          # float32 [B]
    tau: np.ndarray             # float32 [B]
    temp: np.ndarray            # float32 [B]
    uniforms: np.ndarray        # float32 [S, B]
    k_new: Optional[np.ndarray]  # [S, B, Hkv, d] appended keys (closed loop)
    v_new: Optional[np.ndarray]  # [S, B, Hkv, d]
    planted: Optional[np.ndarray]  # int64 [B] offset of the planted run, -1 if none

    @property
    def steps(self) -> int:
        return self.logits.shape[0]


def _ctx_lengths(w: Workload, rng: np.random.Generator) -> np.ndarray:
    kind = w.ctx[0]
    if kind == "uniform":
        lo, hi = w.ctx[1], w.ctx[2]
        return rng.integers(lo, hi + 1, size=w.batch).astype(np.int32)
    if kind == "lognormal":
        median, sigma, lo, hi = w.ctx[1:]
        x = rng.lognormal(mean=math.log(median), sigma=sigma, size=w.batch)
        return np.clip(np.rint(x), lo, hi).astype(np.int32)
    if kind == "fixed":
        return np.asarray(w.ctx[1], dtype=np.int32).reshape(w.batch)
    raise ValueError(kind)


def generate(w: Workload, seed: Optional[int] = None, ctx_lens=None) -> Inputs:
    """All inputs of workload `w` (every step of a closed loop).

    `ctx_lens` overrides the drawn context lengths (edge-case tests)."""
    root = np.random.SeedSequence(SEED_BASE + w.index if seed is None else seed)
    children = root.spawn(1 + w.batch)
    g = np.random.default_rng(children[0])
    B, S, V = w.batch, w.steps, w.vocab
    Hq, Hkv, d, bs = w.num_q_heads, w.num_kv_heads, w.head_dim, w.block_size

    drawn = _ctx_lengths(w, g)
    ctx = drawn if ctx_lens is None else np.asarray(ctx_lens, dtype=np.int32).reshape(B)
    scales = g.uniform(w.logit_scale[0], w.logit_scale[1], size=B)
    h_prev = g.uniform(0.0, math.log(V), size=B).astype(np.float32)
    uniforms = g.random(size=(S, B), dtype=np.float32)
    appended = S if S > 1 else 0            # every step of a closed loop appends its token
    nb_alloc = (ctx.astype(np.int64) + appended + bs - 1) // bs
    P = int(nb_alloc.sum())
    perm = g.permutation(P).astype(np.int32)
    drift = g.normal(0.0, w.drift_sigma, size=(max(S - 1, 0), B)) if S > 1 else None

    maxb = w.max_blocks_per_seq
    if int(nb_alloc.max(initial=0)) > maxb:
        raise ValueError("context exceeds the workload's maximum blocks per sequence")
    tables = np.full((B, maxb), -1, dtype=np.int32)
    offs = np.concatenate([[0], np.cumsum(nb_alloc)])
    for s in range(B):
        tables[s, :nb_alloc[s]] = perm[offs[s]:offs[s + 1]]

    # Per-step logit scale (closed loop: reflected walk).
    svals = np.empty((S, B), dtype=np.float64)
    svals[0] = scales
    lo, hi = w.logit_scale
    for t in range(1, S):
        x = svals[t - 1] + drift[t - 1]
        for _ in range(4):
            x = np.where(x < lo, 2 * lo - x, x)
            x = np.where(x > hi, 2 * hi - x, x)
        svals[t] = np.clip(x, lo, hi)

    bf = w.kv_dtype == "bf16"
    edt = np.uint16 if bf else np.float32
    k_pool = np.empty((P, Hkv, bs, d), dtype=edt)
    v_pool = np.empty((P, Hkv, d, bs), dtype=edt)
    q = np.empty((S, B, Hq, d), dtype=edt)
    logits = np.empty((S, B, V), dtype=np.float32)
    k_new = np.empty((S, B, Hkv, d), dtype=edt) if S > 1 else None
    v_new = np.empty((S, B, Hkv, d), dtype=edt) if S > 1 else None
    planted = np.full(B, -1, dtype=np.int64)

    for s in range(B):
        r = np.random.default_rng(children[1 + s])
        nb = int(nb_alloc[s])
        phys = tables[s, :nb]
        q[:, s] = _normal_values(r, (S, Hq, d), w.kv_dtype)
        kt = _normal_values(r, (nb, Hkv, bs, d), w.kv_dtype)
        vt = _normal_values(r, (nb, Hkv, d, bs), w.kv_dtype)
        if w.planted_run and int(ctx[s]) >= w.planted_run:
            off = int(r.integers(0, int(ctx[s]) - w.planted_run + 1))
            planted[s] = off
            _plant_run(w, r, q[0, s], kt, off)
        k_pool[phys] = kt
        v_pool[phys] = vt
        for t in range(S):
            logits[t, s] = _logit_row(w, r, s, svals[t, s])
        if S > 1:
            k_new[:, s] = _normal_values(r, (S, Hkv, d), w.kv_dtype)
            v_new[:, s] = _normal_values(r, (S, Hkv, d), w.kv_dtype)

    return Inputs(
        workload=w, ctx_lens=ctx, block_tables=tables, num_pool_blocks=P,
        k_pool=k_pool, v_pool=v_pool, q=q, logits=logits, h_prev=h_prev,
        tau=np.zeros(B, dtype=np.float32), temp=np.full(B, 1.0, dtype=np.float32),
        uniforms=uniforms, k_new=k_new, v_new=v_new, planted=planted)


def _logit_row(w: Workload, r: np.random.Generator, s: int, scale: float) -> np.ndarray:
    V = w.vocab
    if w.logits == "zipf_flat":
        if s % 2 == 0:
            ranks = r.permutation(V).astype(np.float64) + 1.0
            return (-ZIPF_EXPONENT * np.log(ranks)).astype(np.float32)
        return (r.standard_normal(V, dtype=np.float32) * np.float32(w.logit_scale[0]))
    return r.standard_normal(V, dtype=np.float32) * np.float32(scale)


def _plant_run(w: Workload, r: np.random.Generator, q_bits: np.ndarray, kt: np.ndarray,
               off: int) -> None:
    """Overwrite keys of tokens off..off+run-1 with a run close to each group's mean query."""
    G, d, bs = w.group, w.head_dim, w.block_size
    qf = bf16_bits_to_f32(q_bits).astype(np.float64) if w.kv_dtype == "bf16" \
        else q_bits.astype(np.float64)
    c = w.planted_cos
    for g in range(w.num_kv_heads):
        u = qf[g * G:(g + 1) * G].mean(axis=0)
        u /= np.linalg.norm(u)
        wv = r.standard_normal((w.planted_run, d))
        wv -= np.outer(wv @ u, u)
        wv /= np.linalg.norm(wv, axis=1, keepdims=True)
        keys = math.sqrt(d) * (c * u[None, :] + math.sqrt(1.0 - c * c) * wv)
        keys = keys.astype(np.float32)
        vals = f32_to_bf16_bits(keys) if w.kv_dtype == "bf16" else keys
        for i in range(w.planted_run):
            tok = off + i
            kt[tok // bs, g, tok % bs, :] = vals[i]
