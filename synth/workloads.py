"""Shapes and value recipes of the synthetic decode-step workloads.

Each workload is one batched decode step (or a closed loop of steps) of
entropic-time inference: a batch of sequences, each with a paged KV cache,
one query vector per head and one next-token logit row.  The paper measures
on an unnamed pretrained decoder and an unnamed prompt mixture (Section 6,
"Experimental Setup"); these seeded synthetic workloads stand in for them.

This module holds shapes and recipes only: no arithmetic of the method.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass
from typing import Optional, Tuple

SEED_BASE = 2603033100


@dataclass(frozen=True)
class Workload:
    name: str
    index: int                    # seed offset: seed = SEED_BASE + index
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    kv_dtype: str                 # "f32" or "bf16" (queries use the same dtype)
    vocab: int
    ctx: Tuple                    # ("uniform", lo, hi) | ("lognormal", median, sigma, lo, hi)
                                  # | ("fixed", [lengths])
    logits: str                   # "normal" | "zipf_flat"
    logit_scale: Tuple[float, float]   # U[lo, hi] of the per-sequence logit std
    h_target: float
    block_size: int = 16
    steps: int = 1                # decode steps (closed loop when > 1)
    planted_run: int = 0          # tokens of the planted high-similarity key run (0 = none)
    planted_cos: float = 0.9
    drift_sigma: float = 0.0      # per-step N(0, sigma^2) walk of the logit scale (closed loop)

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def ctx_max(self) -> int:
        if self.ctx[0] == "uniform":
            return int(self.ctx[2])
        if self.ctx[0] == "fixed":
            return int(max(self.ctx[1]))
        return int(self.ctx[4])

    @property
    def max_blocks_per_seq(self) -> int:
        """Logical blocks a sequence can reach, appended tokens included."""
        return -(-(self.ctx_max + (self.steps if self.steps > 1 else 0)) // self.block_size)

    @property
    def elem_bytes(self) -> int:
        return 2 if self.kv_dtype == "bf16" else 4

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads.  Sizes follow the decode configurations the build is
# measured on; value recipes for details those configurations leave open are
# stated next to each field.
TINY = Workload(
    name="tiny", index=0, batch=4, num_q_heads=8, num_kv_heads=8, head_dim=64,
    kv_dtype="f32", vocab=1024, ctx=("uniform", 128, 512), logits="normal",
    logit_scale=(0.5, 4.0), h_target=2.0)

LLAMA3_8B = Workload(
    name="llama3_8b_decode", index=1, batch=64, num_q_heads=32, num_kv_heads=8,
    head_dim=128, kv_dtype="bf16", vocab=128256, ctx=("uniform", 2048, 8192),
    logits="normal", logit_scale=(0.5, 4.0), h_target=2.5)

LONG_CONTEXT = Workload(
    name="long_context", index=2, batch=16, num_q_heads=32, num_kv_heads=8,
    head_dim=128, kv_dtype="bf16", vocab=128256, ctx=("uniform", 32768, 131072),
    logits="normal", logit_scale=(0.5, 4.0), h_target=2.5, planted_run=64)

SKEWED = Workload(
    name="skewed_mixed", index=3, batch=256, num_q_heads=32, num_kv_heads=8,
    head_dim=128, kv_dtype="bf16", vocab=128256,
    ctx=("lognormal", 1024, 1.0, 64, 32768), logits="zipf_flat",
    logit_scale=(0.3, 0.3), h_target=2.5)

LLAMA70B_LOOP = Workload(
    name="llama70b_closed_loop", index=4, batch=128, num_q_heads=64, num_kv_heads=8,
    head_dim=128, kv_dtype="bf16", vocab=128256, ctx=("uniform", 4096, 16384),
    logits="normal", logit_scale=(0.3, 5.0), h_target=2.5, steps=64,
    drift_sigma=0.25)

WORKLOADS = {w.name: w for w in (TINY, LLAMA3_8B, LONG_CONTEXT, SKEWED, LLAMA70B_LOOP)}

# Zipf exponent of the peaked half of the skewed batch.
ZIPF_EXPONENT = 1.2


def small(w: Workload, batch: int, ctx: Optional[Tuple] = None, vocab: Optional[int] = None,
          steps: Optional[int] = None, suffix: str = "small") -> Workload:
    """A reduced copy of `w` (same head shapes and dtype) for fast parity tests."""
    kw = dict(batch=batch, name=f"{w.name}_{suffix}")
    if ctx is not None:
        kw["ctx"] = ctx
    if vocab is not None:
        kw["vocab"] = vocab
    if steps is not None:
        kw["steps"] = steps
    return w.replace(**kw)

