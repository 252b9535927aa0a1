"""GPU parity of the top-k and tail-corrected entropy estimators (Section 2.1)
and of the controller and guarded block budget acting on them (Section 3.3),
through the C ABI, against the float64 oracle.

Cases: the 8B-shaped batch (thread maxima staged in LDS), a vocabulary above
131072 (thread maxima read from memory), rows with ties at every level,
uniform, one-hot and partly masked rows, k >= |V| (the exact entropy), k = 1,
the long-table selection (block tables over 1024 blocks), and a
closed loop with a positive estimator error bound in the budget.  The fused
step must give exactly the outputs of the four per-stage calls.
"""
import math

import numpy as np
import pytest

from oracle import entropy as OE
from synth import LLAMA3_8B, LLAMA70B_LOOP, LONG_CONTEXT, SKEWED, TINY, default_params, generate, small
from tests.test_gpu_parity import _assert_ok, _run, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

TOPK, TAIL = OE.TOPK, OE.TAIL
FIELDS = ("h", "tau", "temp", "temp_used", "row_stats", "kept", "n_kept", "scores", "theta",
          "out", "lse", "tokens")


def _both(torch, w, p, x=None, steps=1):
    """Fused and staged runs of the same inputs; parity of both, and the
    fused outputs equal the staged ones bit for bit."""
    x = generate(w) if x is None else x
    reps_f, df = _run(torch, x, p, fused=True, steps=steps)
    _assert_ok(reps_f)
    x2 = generate(w)
    if x is not None:
        x2.logits[...] = x.logits
        x2.h_prev[...] = x.h_prev
    reps_s, ds = _run(torch, x2, p, fused=False, steps=steps)
    _assert_ok(reps_s)
    for name in FIELDS:
        a, b = getattr(df, name).cpu().numpy(), getattr(ds, name).cpu().numpy()
        assert np.array_equal(a, b, equal_nan=True), name
    return df


@pytest.mark.parametrize("est", [TOPK, TAIL], ids=["topk", "tail"])
@pytest.mark.parametrize("k", [1, 50, 256, 512])
def test_llama3_8b_small(torch_cuda, est, k):
    w = small(LLAMA3_8B, 4, ctx=("uniform", 100, 1500), suffix=f"est{est}_{k}")
    p = default_params(w).replace(estimator=est, est_k=k)
    _both(torch_cuda, w, p)


@pytest.mark.parametrize("est", [TOPK, TAIL], ids=["topk", "tail"])
def test_tiny_and_k_at_least_vocab(torch_cuda, est):
    """Tiny (|V| = 1024, fp32 KV): k = 256, and k = 512; with k >= |V| the
    estimate is the exact entropy."""
    for k in (256, 512):
        _both(torch_cuda, TINY, default_params(TINY).replace(estimator=est, est_k=k))
    w = small(TINY, 4, vocab=300, suffix="v300")
    p = default_params(w).replace(estimator=est, est_k=300)
    df = _both(torch_cuda, w, p)
    x = generate(w)
    h = df.h.cpu().numpy()
    for s in range(w.batch):
        assert abs(h[s] - OE.entropy(x.logits[0, s], float(x.temp[s]))) < 1e-4


def test_large_vocab_maxima_from_memory(torch_cuda):
    """|V| = 200000: 49 chunks, 12544 thread maxima (read from memory)."""
    w = small(SKEWED, 6, ctx=("uniform", 64, 900), vocab=200000, suffix="v200k")
    p = default_params(w).replace(estimator=TAIL, est_k=300)
    _both(torch_cuda, w, p)


@pytest.mark.parametrize("est", [TOPK, TAIL], ids=["topk", "tail"])
def test_ties_uniform_onehot_masked_rows(torch_cuda, est):
    w = small(SKEWED, 8, ctx=("uniform", 40, 400), vocab=5000, suffix=f"estedge{est}")
    x = generate(w)
    V = w.vocab
    rng = np.random.default_rng(5)
    x.logits[0, 0] = 0.5                                             # uniform
    x.logits[0, 1] = 0.0
    x.logits[0, 1, 4321] = 1000.0                                    # one-hot
    x.logits[0, 2] = rng.integers(0, 4, V).astype(np.float32)        # ties at every level
    x.logits[0, 3, : V // 2] = -np.inf                               # half masked
    x.logits[0, 4] = -np.inf
    x.logits[0, 4, [3, 4097, 4999]] = 1.25                           # three finite, tied
    x.logits[0, 5, ::7] = 3.0                                        # many ties at the top
    k = 64
    p = default_params(w).replace(estimator=est, est_k=k)
    df = _both(torch_cuda, w, p, x=x)
    h = df.h.cpu().numpy()
    if est == TOPK:
        assert abs(h[0] - math.log(k)) < 1e-4
        assert abs(h[1]) < 1e-6
    else:
        # Uniform row: H~ = ln k, mbar = 1 - k/|V|, and the estimate exceeds
        # ln |V| by mbar ln k (H~ enters with weight 1, not m).
        mbar = 1.0 - k / V
        hb = -mbar * math.log(mbar) - (1 - mbar) * math.log1p(-mbar)
        assert abs(h[0] - (math.log(k) + hb + mbar * math.log(V - k))) < 1e-4
        assert abs(h[0] - math.log(V) - mbar * math.log(k)) < 1e-4
    assert abs(h[4] - math.log(3)) < 1e-4                            # fewer finite logits than k


def test_three_launch_selection(torch_cuda):
    """Block tables over 1024 blocks: the entropy estimate and the controller
    in the fused step's tile launch (whose selecting workgroup, when it is
    the entropy one, reuses the estimator's LDS for its keys) and in the
    first of the staged form's three selection launches; both forms equal
    bit for bit."""
    w = small(LONG_CONTEXT, 3, ctx=("uniform", 9000, 20000), suffix="est_long")
    p = default_params(w).replace(estimator=TAIL, est_k=256)
    _both(torch_cuda, w, p)


def test_closed_loop_guarded_budget(torch_cuda):
    """Four steps with appends; the controller acts on the tail-corrected
    estimate and the budget adds its error bound eps_H (the safety floor of
    Section 3.3)."""
    w = small(LLAMA70B_LOOP, 3, ctx=("uniform", 100, 600), steps=4, suffix="est_loop")
    p = default_params(w).replace(estimator=TAIL, est_k=128, eps_h=0.25)
    x = generate(w)
    reps, dev = _run(torch_cuda, x, p, steps=4)
    _assert_ok(reps)
