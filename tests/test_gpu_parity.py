"""GPU parity of the whole decode step against the float64 oracle, through the C ABI.

Teacher-forced per stage (see tests/parity.py for the bands).  Workloads:
Tiny (fp32), reduced bf16 variants of the Llama-3-8B, long-context (planted
run), skewed and 70B-shaped configurations that still span several tiles and
ragged tails, edge cases (empty, one-token and partial blocks; uniform,
one-hot and masked logit rows), keep-all equals dense attention, a closed
loop with appends, and the full-size Llama-3-8B step on sampled sequences.
"""
import math

import numpy as np
import pytest

from synth import (LLAMA3_8B, LLAMA70B_LOOP, LONG_CONTEXT, SKEWED, TINY, default_params, generate,
                   small)
from synth.device import config_fields, upload
from tests.parity import Report, check_step, collect, run_step

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2603_03310_amd import ent
    ent.load()          # raises if the library is missing: no fallback
    return torch


def _run(torch, x, p, steps=1, seqs=None, max_blocks=None, check_ksum=True, fused=True):
    from paper_2603_03310_amd.runner import Decoder
    w = x.workload
    dev = upload(x)
    reps = []
    with Decoder(**config_fields(w, p, x.num_pool_blocks, max_blocks=max_blocks)) as dec:
        B = w.batch
        dec.summarize(B, dev.k_pool, dev.block_tables, dev.ctx_lens, dev.ksum)
        kp, vp = x.k_pool.copy(), x.v_pool.copy()
        ctx = x.ctx_lens.copy()
        for t in range(steps):
            state = (dev.h_prev.cpu().numpy().copy(), dev.tau.cpu().numpy().copy(),
                     dev.temp.cpu().numpy().copy())
            run_step(dec, dev, t, fused=fused)
            torch.cuda.synchronize()
            gpu = collect(dev)
            print(f"[parity] {w.name} step {t}: kept fraction "
                  f"{gpu.n_kept.sum() / max(1, sum(-(-int(n) // 16) for n in ctx)):.3f}",
                  flush=True)
            rep = check_step(k_pool=kp, v_pool=vp, tables=x.block_tables, ctx_lens=ctx, q=x.q[t],
                             logits=x.logits[t], uniforms=x.uniforms[t], h_prev=state[0],
                             tau=state[1], temp=state[2], params=p, gpu=gpu, seqs=seqs,
                             check_ksum=check_ksum)
            print(f"[parity] {w.name} step {t}: score err {rep.max_score_err:.2e} "
                  f"(rel {rep.max_score_rel_err:.2e}), attention err {rep.max_att_err:.2e}, "
                  f"entropy err {rep.max_h_err:.2e}", flush=True)
            reps.append(rep)
            if steps > 1:
                dec.append(B, dev.k_new[t], dev.v_new[t], dev.block_tables, dev.ctx_lens,
                           dev.k_pool, dev.v_pool, dev.ksum)
                from oracle import append as OAp
                for s in range(B):
                    ctx[s] = OAp.append_token(kp, vp, x.block_tables[s], int(ctx[s]),
                                              x.k_new[t, s], x.v_new[t, s], 16)
        flags = dec.device_status()
    assert flags == 0, f"device flags {flags}"
    return reps, dev


def _assert_ok(reps):
    for i, r in enumerate(reps):
        assert r.ok(), f"step {i}: " + "; ".join(r.failures[:8])


def test_tiny(torch_cuda):
    x = generate(TINY)
    reps, _ = _run(torch_cuda, x, default_params(TINY))
    _assert_ok(reps)


BF16_SMALL = [
    small(LLAMA3_8B, 3, ctx=("uniform", 100, 1500)),
    small(LONG_CONTEXT, 2, ctx=("uniform", 3000, 9000)),
    small(SKEWED, 12, ctx=("lognormal", 300, 1.0, 1, 3000)),
    small(LLAMA70B_LOOP, 3, ctx=("uniform", 100, 700), steps=1),
]


@pytest.mark.parametrize("w", BF16_SMALL, ids=lambda w: w.name)
def test_bf16_small(torch_cuda, w):
    x = generate(w)
    reps, _ = _run(torch_cuda, x, default_params(w))
    _assert_ok(reps)


def test_edge_contexts_and_logit_rows(torch_cuda):
    w = small(SKEWED, 10, ctx=("fixed", [0, 1, 15, 16, 17, 33, 64, 65, 100, 1000]), vocab=5000,
              suffix="edge")
    x = generate(w)
    V = w.vocab
    x.logits[0, 0] = 0.5                                   # uniform: H = log V
    x.logits[0, 1] = 0.0
    x.logits[0, 1, 4321] = 1000.0                          # one-hot: H = 0
    x.logits[0, 2] = -np.inf
    x.logits[0, 2, [3, 4097, 4999]] = 1.25                 # three tied finite logits: H = log 3
    x.logits[0, 3, : V // 2] = -np.inf                     # half the vocabulary masked
    x.h_prev[4] = np.nan                                   # no previous step
    p = default_params(w)
    reps, dev = _run(torch_cuda, x, p)
    _assert_ok(reps)
    h = dev.h.cpu().numpy()
    assert abs(h[0] - math.log(V)) < 1e-4 and abs(h[1]) < 1e-6 and abs(h[2] - math.log(3)) < 1e-4
    assert dev.tau.cpu().numpy()[4] == 0.0
    assert int(dev.n_kept.cpu().numpy()[0]) == 0            # empty sequence keeps nothing
    assert np.all(dev.out.cpu().numpy()[0] == 0)
    assert int(dev.tokens.cpu().numpy()[1]) == 4321
    assert int(dev.tokens.cpu().numpy()[2]) in (3, 4097, 4999)


def test_keep_all_equals_dense(torch_cuda):
    w = small(LLAMA3_8B, 3, ctx=("uniform", 200, 900), suffix="dense")
    x = generate(w)
    p = default_params(w).replace(kappa_min=1.0)
    reps, dev = _run(torch_cuda, x, p)
    _assert_ok(reps)
    nk = dev.n_kept.cpu().numpy()
    assert list(nk) == [-(-int(n) // 16) for n in x.ctx_lens]


def test_temperature_unchanged_at_target(torch_cuda):
    # Run once to learn the GPU entropy, then make it the target: T must not move.
    w = small(LLAMA3_8B, 2, ctx=("uniform", 50, 200), suffix="target")
    x = generate(w)
    p = default_params(w)
    _, dev = _run(torch_cuda, x, p)
    h = dev.h.cpu().numpy()
    for s in range(2):
        x1 = generate(w)
        p1 = p.replace(h_target=float(h[s]))
        _, dev1 = _run(torch_cuda, x1, p1)
        assert dev1.h.cpu().numpy()[s] == h[s]
        assert dev1.temp.cpu().numpy()[s] == np.float32(x1.temp[s])


@pytest.mark.parametrize("fused", [True, False], ids=["fused", "staged"])
def test_closed_loop_with_appends(torch_cuda, fused):
    w = small(LLAMA70B_LOOP, 4, ctx=("uniform", 100, 600), steps=6)
    x = generate(w)
    reps, dev = _run(torch_cuda, x, default_params(w), steps=6, fused=fused)
    _assert_ok(reps)
    assert list(dev.ctx_lens.cpu().numpy()) == list(x.ctx_lens + 6)


@pytest.mark.parametrize("w", [small(LLAMA70B_LOOP, 4, ctx=("uniform", 100, 600), steps=6,
                                     suffix="refresh"),
                               small(TINY, TINY.batch, steps=6, suffix="refresh")],
                         ids=lambda w: w.name)
def test_append_refresh_matches_fresh_summary(torch_cuda, w):
    """The mean keys that appends keep up to date equal, bit for bit, the
    ones a fresh summary pass computes over the grown cache (both sum a
    block's slots in slot order), for bf16 and fp32 caches; every step is
    checked against the oracle on the way."""
    from paper_2603_03310_amd.runner import Decoder
    x = generate(w)
    p = default_params(w)
    reps, dev = _run(torch_cuda, x, p, steps=6)
    _assert_ok(reps)
    fresh = torch_cuda.zeros_like(dev.ksum)
    with Decoder(**config_fields(w, p, x.num_pool_blocks)) as dec:
        dec.summarize(w.batch, dev.k_pool, dev.block_tables, dev.ctx_lens, fresh)
        torch_cuda.cuda.synchronize()
        assert dec.device_status() == 0
    a, b = dev.ksum.cpu().numpy(), fresh.cpu().numpy()
    ctx = dev.ctx_lens.cpu().numpy()
    for s in range(w.batch):
        phys = np.asarray(x.block_tables[s][: -(-int(ctx[s]) // 16)], dtype=np.int64)
        assert np.array_equal(a[phys], b[phys]), f"seq {s}"


FUSED_CASES = [
    TINY,
    small(LLAMA3_8B, 5, ctx=("uniform", 100, 2500), suffix="fused"),
    # more than 1024 blocks per table row: the long-table selection
    small(LONG_CONTEXT, 3, ctx=("uniform", 9000, 20000), suffix="fused_long"),
    small(SKEWED, 10, ctx=("fixed", [0, 1, 15, 16, 17, 33, 64, 65, 100, 1000]), vocab=5000,
          suffix="fused_edge"),
]


@pytest.mark.parametrize("w", FUSED_CASES, ids=lambda w: w.name)
def test_fused_step_matches_staged(torch_cuda, w):
    """ent_decode_step gives exactly the outputs of the four per-stage calls."""
    x = generate(w)
    p = default_params(w)
    reps_f, df = _run(torch_cuda, x, p, fused=True)
    _assert_ok(reps_f)
    _, ds = _run(torch_cuda, generate(w), p, fused=False)
    for name in ("h", "tau", "temp", "temp_used", "row_stats", "kept", "n_kept", "scores",
                 "theta", "out", "lse", "tokens"):
        a, b = getattr(df, name).cpu().numpy(), getattr(ds, name).cpu().numpy()
        assert np.array_equal(a, b, equal_nan=True), name


def test_deterministic(torch_cuda):
    w = small(LLAMA3_8B, 4, ctx=("uniform", 500, 3000), suffix="det")
    x = generate(w)
    _, d1 = _run(torch_cuda, x, default_params(w), check_ksum=False)
    _, d2 = _run(torch_cuda, generate(w), default_params(w), check_ksum=False)
    for name in ("h", "tau", "temp", "kept", "n_kept", "scores", "out", "lse", "tokens"):
        a, b = getattr(d1, name).cpu().numpy(), getattr(d2, name).cpu().numpy()
        assert np.array_equal(a, b, equal_nan=True), name


def test_full_size_llama3_8b_sampled(torch_cuda):
    x = generate(LLAMA3_8B)
    rng = np.random.default_rng(0)
    seqs = sorted(rng.choice(LLAMA3_8B.batch, size=6, replace=False).tolist())
    print(f"[parity] full-size llama3_8b_decode, sampled sequences {seqs}", flush=True)
    reps, dev = _run(torch_cuda, x, default_params(LLAMA3_8B), seqs=seqs)
    _assert_ok(reps)


def _sampled(batch, n, seed):
    rng = np.random.default_rng(seed)
    return sorted(rng.choice(batch, size=min(n, batch), replace=False).tolist())


def test_full_size_long_context_sampled(torch_cuda):
    """Full long-context step (B=16, N up to 131072): parity on two sampled
    sequences, and the planted high-similarity run's full blocks outrank the
    rest: they are kept whenever the budget covers them."""
    x = generate(LONG_CONTEXT)
    seqs = _sampled(LONG_CONTEXT.batch, 2, 1)
    print(f"[parity] full-size long_context, sampled sequences {seqs}", flush=True)
    reps, dev = _run(torch_cuda, x, default_params(LONG_CONTEXT), seqs=seqs)
    _assert_ok(reps)
    scores = dev.scores.cpu().numpy()
    n_kept = dev.n_kept.cpu().numpy()
    kept = dev.kept.cpu().numpy()
    for s in range(LONG_CONTEXT.batch):
        off = int(x.planted[s])
        if off < 0:
            continue
        full = [j for j in range(-(-off // 16), (off + LONG_CONTEXT.planted_run) // 16)]
        nb = -(-int(x.ctx_lens[s]) // 16)
        sc = scores[s, :nb]
        order = np.argsort(-sc, kind="stable")
        # The (up to two) partly planted blocks at the run's ends may rank among them.
        top = len(full) + 2
        assert set(full) <= set(order[:top].tolist()), f"seq {s}: planted blocks not top-ranked"
        if int(n_kept[s]) >= top:
            assert set(full) <= set(kept[s, : int(n_kept[s])].tolist()), f"seq {s}: planted block pruned"


def test_full_size_skewed_sampled(torch_cuda):
    """Full skewed batch (B=256, lognormal contexts, Zipf and flat logit rows)
    on sampled sequences of both logit kinds."""
    x = generate(SKEWED)
    seqs = sorted(set(_sampled(SKEWED.batch, 6, 2)) | {0, 1})
    print(f"[parity] full-size skewed_mixed, sampled sequences {seqs}", flush=True)
    reps, _ = _run(torch_cuda, x, default_params(SKEWED), seqs=seqs)
    _assert_ok(reps)


def test_full_size_70b_loop_three_steps(torch_cuda):
    """70B-shaped batch at full size (B=128, 64/8 heads, N in [4096,16384]):
    three closed-loop steps with appends, parity on sampled sequences."""
    w = small(LLAMA70B_LOOP, LLAMA70B_LOOP.batch, steps=3, suffix="full3")
    x = generate(w)
    seqs = _sampled(w.batch, 4, 3)
    print(f"[parity] full-size llama70b shapes, 3 steps, sampled sequences {seqs}", flush=True)
    reps, dev = _run(torch_cuda, x, default_params(w), steps=3, seqs=seqs)
    _assert_ok(reps)
    assert list(dev.ctx_lens.cpu().numpy()) == list(x.ctx_lens + 3)
