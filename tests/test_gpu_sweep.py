"""A sweep over option combinations (estimator, scoring mode, forced keeps,
calibration and rate guards, budget floors, estimator error bound) and
shapes (fp32 and bf16 caches, head_dim 64 and 128, GQA groups 1 to 16,
short and long block tables, ragged contexts), each a seeded small workload checked against the
oracle in both the one-call step and the staged calls.  The cases are drawn
once from a fixed seed, so the sweep is the same on every run.
"""
import math

import numpy as np
import pytest

from synth import LLAMA3_8B, LLAMA70B_LOOP, LONG_CONTEXT, SKEWED, TINY, default_params, generate, small
from tests.test_gpu_parity import _assert_ok, _run, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu


def _cases(n=42, seed=20261202):
    rng = np.random.default_rng(seed)
    bases = [
        (TINY, lambda: small(TINY, int(rng.integers(1, 6)), ctx=("uniform", 1, 600),
                             suffix="sweep")),
        (LLAMA3_8B, lambda: small(LLAMA3_8B, int(rng.integers(1, 5)), ctx=("uniform", 1, 1400),
                                  suffix="sweep")),
        (SKEWED, lambda: small(SKEWED, int(rng.integers(2, 9)),
                               ctx=("lognormal", 200, 1.0, 1, 2500), vocab=20000, suffix="sweep")),
        (LLAMA70B_LOOP, lambda: small(LLAMA70B_LOOP, int(rng.integers(1, 4)),
                                      ctx=("uniform", 16, 900), steps=1, suffix="sweep")),
        (LONG_CONTEXT, lambda: small(LONG_CONTEXT, 1, ctx=("uniform", 2000, 20000),
                                     suffix="sweep")),
        (LLAMA3_8B, lambda: small(LLAMA3_8B.replace(num_q_heads=16, num_kv_heads=8, head_dim=64),
                                  int(rng.integers(1, 5)), ctx=("uniform", 1, 700),
                                  suffix="sweep_d64g2")),
        (LLAMA3_8B, lambda: small(LLAMA3_8B.replace(num_q_heads=32, num_kv_heads=2),
                                  int(rng.integers(1, 4)), ctx=("uniform", 1, 900),
                                  suffix="sweep_g16")),
    ]
    out = []
    for i in range(n):
        base, make = bases[i % len(bases)]
        w = make()
        seed = int(rng.integers(0, 2**31))
        over = dict(
            estimator=int(rng.integers(0, 3)), est_k=int(rng.choice([1, 16, 256])),
            scoring=int(rng.integers(0, 2)),
            keep_first=int(rng.choice([0, 0, 1, 3])), keep_last=int(rng.choice([0, 0, 1, 2])),
            t_cal=float(rng.choice([1.0, 1.7, 0.6])), rho_t=float(rng.choice([math.inf, 0.1])),
            h_bias=float(rng.choice([0.0, 0.0, -0.7, 0.9])),
            eps_h=float(rng.choice([0.0, 0.3])), b_min=int(rng.choice([0, 4, 16])),
            kappa_min=float(rng.choice([0.0, 0.05, 0.3])))
        out.append((f"{i:02d}-{w.name}", w, seed, over))
    return out


CASES = _cases()


@pytest.mark.parametrize("fused", [True, False], ids=["step", "staged"])
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_option_sweep(torch_cuda, case, fused):
    name, w, seed, over = case
    x = generate(w, seed=seed)
    p = default_params(w).replace(**over)
    print(f"[sweep] {name} seed={seed} {over}", flush=True)
    reps, _ = _run(torch_cuda, x, p, fused=fused)
    _assert_ok(reps)
