"""GPU parity of the exact token-level scoring mode and of the forced keeps
(Section 3.2 block contributions from the exact attention weights; forced
first and last blocks) through the C ABI, against the float64 oracle.
Exact mode: bf16 (MFMA) and fp32 (VALU) caches, short and long block tables
(one-launch and long-table selections), ragged and one-token blocks, the full
long-context batch on sampled sequences, a closed loop with appends, and the
staged calls against the one-call step.  Forced
keeps: mean-key and exact modes, forced sets that fill the budget, both
selection forms.
"""
import numpy as np
import pytest

from synth import LLAMA3_8B, LONG_CONTEXT, SKEWED, TINY, default_params, generate, small
from tests.test_gpu_parity import _assert_ok, _run, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

EXACT = [
    small(LLAMA3_8B, 3, ctx=("uniform", 100, 1500), suffix="exact"),
    small(LONG_CONTEXT, 2, ctx=("uniform", 3000, 9000), suffix="exact"),
    small(SKEWED, 10, ctx=("fixed", [1, 15, 16, 17, 33, 64, 65, 100, 1000, 0]), vocab=5000,
          suffix="exact_edge"),
]


def _report(reps, tag):
    for r in reps:
        print(f"[exact] {tag}: max score error {r.max_score_err:.3g}, "
              f"band-exempt blocks {r.band_exempt}", flush=True)


@pytest.mark.parametrize("fused", [True, False], ids=["step", "staged"])
@pytest.mark.parametrize("w", EXACT, ids=lambda w: w.name)
def test_exact_scoring(torch_cuda, w, fused):
    x = generate(w)
    p = default_params(w).replace(scoring=1)
    reps, _ = _run(torch_cuda, x, p, fused=fused)
    _report(reps, w.name)
    _assert_ok(reps)


def test_exact_full_size_long_context_sampled(torch_cuda):
    """The full long-context batch in exact mode (B=16, N up to 131072: up to
    512 tiles of 16 blocks per sequence, every key of 2.5 GB of K read once),
    parity on three sampled sequences."""
    x = generate(LONG_CONTEXT)
    seqs = sorted(np.random.default_rng(5).choice(LONG_CONTEXT.batch, size=3, replace=False).tolist())
    print(f"[exact] full-size long_context, sampled sequences {seqs}", flush=True)
    reps, _ = _run(torch_cuda, x, default_params(LONG_CONTEXT).replace(scoring=1), seqs=seqs)
    _report(reps, "long_context full")
    _assert_ok(reps)


def test_exact_scoring_fp32(torch_cuda):
    x = generate(TINY)
    reps, _ = _run(torch_cuda, x, default_params(TINY).replace(scoring=1))
    _report(reps, "tiny")
    _assert_ok(reps)


def test_exact_closed_loop_with_appends(torch_cuda):
    w = small(LLAMA3_8B, 3, ctx=("uniform", 30, 200), steps=3, suffix="exact_loop")
    x = generate(w)
    reps, _ = _run(torch_cuda, x, default_params(w).replace(scoring=1), steps=3)
    _assert_ok(reps)


def test_exact_equals_mean_key_on_constant_blocks(torch_cuda):
    """When every token of a block carries the same key, the mean-key
    weights are the exact weights: both modes give the same scores."""
    w = small(LLAMA3_8B, 3, ctx=("fixed", [160, 171, 500]), suffix="constblocks")
    x = generate(w)
    x.k_pool[:] = x.k_pool[:, :, :1, :]          # slot 0's key in every slot of each tile
    scores = []
    for mode in (0, 1):
        _, dev = _run(torch_cuda, x, default_params(w).replace(scoring=mode))
        scores.append(dev.scores.cpu().numpy())
    for s, n in enumerate(x.ctx_lens):
        nb = -(-int(n) // 16)
        np.testing.assert_allclose(scores[1][s, :nb], scores[0][s, :nb], rtol=2e-4, atol=2e-6)


FORCED = [
    small(LLAMA3_8B, 4, ctx=("fixed", [1, 40, 700, 1500]), suffix="forced"),
    small(LONG_CONTEXT, 2, ctx=("uniform", 3000, 9000), suffix="forced"),
]


@pytest.mark.parametrize("keep", [(1, 1), (2, 3), (0, 4)], ids=str)
@pytest.mark.parametrize("fused", [True, False], ids=["step", "staged"])
@pytest.mark.parametrize("w", FORCED, ids=lambda w: w.name)
def test_forced_keeps(torch_cuda, w, fused, keep):
    x = generate(w)
    p = default_params(w).replace(keep_first=keep[0], keep_last=keep[1])
    reps, dev = _run(torch_cuda, x, p, fused=fused)
    _assert_ok(reps)
    kept, nk = dev.kept.cpu().numpy(), dev.n_kept.cpu().numpy()
    for s, n in enumerate(x.ctx_lens):
        nb = -(-int(n) // 16)
        ks = set(kept[s, :nk[s]].tolist())
        assert set(range(min(keep[0], nb))) <= ks
        assert set(range(max(nb - keep[1], 0), nb)) <= ks


def test_forced_keeps_fill_the_budget(torch_cuda):
    """Low entropy and no minimum: the budget is smaller than the forced set,
    which is then exactly what is kept (threshold +inf)."""
    w = small(LLAMA3_8B, 3, ctx=("fixed", [300, 640, 1000]), suffix="forcedfill")
    x = generate(w)
    p = default_params(w).replace(kappa_min=0.0, b_min=0, h_min=20.0, log_v=21.0,
                                  keep_first=3, keep_last=2)
    reps, dev = _run(torch_cuda, x, p)
    _assert_ok(reps)
    nk = dev.n_kept.cpu().numpy()
    assert list(nk) == [5, 5, 5]
    assert np.all(np.isinf(dev.theta.cpu().numpy()))


def test_forced_keeps_with_exact_scoring(torch_cuda):
    w = small(LLAMA3_8B, 3, ctx=("uniform", 100, 1500), suffix="forcedexact")
    x = generate(w)
    p = default_params(w).replace(scoring=1, keep_first=1, keep_last=1)
    for fused in (True, False):
        reps, _ = _run(torch_cuda, x, p, fused=fused)
        _assert_ok(reps)
