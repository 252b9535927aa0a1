"""End-to-end, free-running parity and checkpoint/resume of the closed loop.

Free-running: the oracle computes every stage from the raw inputs alone
(its own entropy, block summaries, scores, kept sets, attention and tokens,
its own controller state carried from step to step) and is compared with
the GPU step by step.  Where a discrete decision lies inside a tie band (an
oracle score within 1e-6 of its threshold, the fp32 budget at a step of the
entropy, a token's CDF margin below 1e-6) the case is reported and the
dependent outputs are not compared; such cases must stay rare.

Checkpoint/resume: the step's state is the caller's arrays (controller
state, kept-fraction state, lengths, K/V pool, block summaries); the
context holds none.  A run interrupted after some steps, saved to the host,
restored into fresh buffers and a fresh context, and resumed must match the
uninterrupted run bit for bit.
"""
import math

import numpy as np
import pytest

from oracle import append as OAp
from oracle import blocks as OB
from oracle import step as OS
from synth import LLAMA3_8B, LLAMA70B_LOOP, SKEWED, TINY, default_params, generate, small
from synth.device import config_fields, upload
from tests.parity import collect, run_step
from tests.test_gpu_parity import torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

BAND = 1e-6
H_TOL = 1e-4
ATT_ABS = ATT_REL = 2e-3


def _compare(o, gpu, s, p, nb, stats, kappa_prev=math.nan):
    """Free-running comparison of sequence s (kappa_prev: the kept-fraction
    state the oracle's step used); returns failure messages."""
    f = []
    for name, gv in (("h", gpu.h[s]), ("tau", gpu.tau[s]), ("temp_next", gpu.temp_next[s])):
        if abs(float(gv) - o[name]) > H_TOL:
            f.append(f"seq {s}: {name} {gv} vs {o[name]}")
    if nb == 0:
        return f
    # Budget boundary: the fp32 budget from the GPU's entropy.
    k_g = OB.keep_budget(float(gpu.h[s]), nb, p, kappa_prev)
    scores = o["scores"]
    theta = o["theta"]
    # Another block's score within the band of the threshold (the block at
    # the threshold itself is always within it).
    near = math.isfinite(theta) and int(np.sum(np.abs(scores - theta) <= BAND)) > 1
    kept_g = gpu.kept[s][: int(gpu.n_kept[s])].tolist()
    if k_g != o["k"] or near:
        stats["band"] += 1
        return f
    if kept_g != o["kept"].tolist():
        f.append(f"seq {s}: kept lists differ outside the tie band")
        return f
    err = np.abs(gpu.out[s].astype(np.float64) - o["o"])
    if np.any(err > ATT_ABS + ATT_REL * np.abs(o["o"])):
        f.append(f"seq {s}: attention differs by {err.max():.3g}")
    if int(gpu.tokens[s]) != o["token"]:
        if o["margin"] < BAND:
            stats["band"] += 1
        else:
            f.append(f"seq {s}: token {gpu.tokens[s]} vs {o['token']}")
    stats["compared"] += 1
    return f


@pytest.mark.parametrize("w", [TINY, small(LLAMA3_8B, 4, ctx=("uniform", 100, 1500), suffix="free"),
                               small(SKEWED, 8, ctx=("lognormal", 300, 1.0, 1, 3000),
                                     suffix="free")], ids=lambda w: w.name)
def test_free_running_step(torch_cuda, w):
    from paper_2603_03310_amd.runner import Decoder
    torch = torch_cuda
    x = generate(w)
    p = default_params(w)
    dev = upload(x)
    with Decoder(**config_fields(w, p, x.num_pool_blocks)) as dec:
        dec.summarize(w.batch, dev.k_pool, dev.block_tables, dev.ctx_lens, dev.ksum)
        run_step(dec, dev, 0)
        torch.cuda.synchronize()
        assert dec.device_status() == 0
    gpu = collect(dev)
    stats = {"band": 0, "compared": 0}
    fails = []
    for s in range(w.batch):
        o = OS.sequence_step(s, k_pool=x.k_pool, v_pool=x.v_pool, tables=x.block_tables,
                             ctx_lens=x.ctx_lens, q=x.q[0], logits=x.logits[0], h_prev=x.h_prev,
                             tau=x.tau, temp=x.temp, uniforms=x.uniforms[0], params=p,
                             block_size=16)
        fails += _compare(o, gpu, s, p, o["nb"], stats)
    print(f"[free] {w.name}: {stats}", flush=True)
    assert not fails, "; ".join(fails[:8])
    assert stats["band"] <= max(1, w.batch // 4)


def test_free_running_closed_loop(torch_cuda):
    """Five steps of the 70B-shaped loop with appends and the guards (rate
    bounds on T and kappa, kept-fraction state), oracle state carried by
    the oracle itself."""
    from paper_2603_03310_amd.runner import Decoder
    torch = torch_cuda
    w = small(LLAMA70B_LOOP, 3, ctx=("uniform", 100, 900), steps=5, suffix="free")
    x = generate(w)
    p = default_params(w).replace(rho_t=0.2, dkappa=0.1)
    dev = upload(x)
    kp, vp, ctx = x.k_pool.copy(), x.v_pool.copy(), x.ctx_lens.copy()
    h_prev, tau, temp = x.h_prev.copy(), x.tau.copy(), x.temp.copy()
    kappa = np.full(w.batch, np.nan)
    stats = {"band": 0, "compared": 0}
    fails = []
    with Decoder(**config_fields(w, p, x.num_pool_blocks)) as dec:
        B = w.batch
        dec.summarize(B, dev.k_pool, dev.block_tables, dev.ctx_lens, dev.ksum)
        for t in range(w.steps):
            run_step(dec, dev, t, kappa=True)
            torch.cuda.synchronize()
            gpu = collect(dev, with_kappa=True)
            outs = [OS.sequence_step(s, k_pool=kp, v_pool=vp, tables=x.block_tables, ctx_lens=ctx,
                                     q=x.q[t], logits=x.logits[t], h_prev=h_prev, tau=tau,
                                     temp=temp, uniforms=x.uniforms[t], params=p, block_size=16,
                                     kappa=kappa) for s in range(B)]
            for s, o in enumerate(outs):
                fails += [f"step {t}: {m}"
                          for m in _compare(o, gpu, s, p, o["nb"], stats, float(kappa[s]))]
            # The oracle carries its own state to the next step.
            h_prev = np.array([o["h"] for o in outs])
            tau = np.array([o["tau"] for o in outs])
            temp = np.array([o["temp_next"] for o in outs])
            kappa = np.array([o["kappa"] for o in outs])
            dec.append(B, dev.k_new[t], dev.v_new[t], dev.block_tables, dev.ctx_lens, dev.k_pool,
                       dev.v_pool, dev.ksum)
            for s in range(B):
                ctx[s] = OAp.append_token(kp, vp, x.block_tables[s], int(ctx[s]), x.k_new[t, s],
                                          x.v_new[t, s], 16)
        assert dec.device_status() == 0
    print(f"[free loop] {stats}", flush=True)
    assert not fails, "; ".join(fails[:8])
    assert stats["band"] <= 2


def _host(t):
    import torch
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16).copy()
    return t.cpu().numpy().copy()


def _run_steps(torch, dec, dev, t0, t1):
    outs = []
    for t in range(t0, t1):
        run_step(dec, dev, t, kappa=True)
        dec.append(dev.ctx_lens.shape[0], dev.k_new[t], dev.v_new[t], dev.block_tables,
                   dev.ctx_lens, dev.k_pool, dev.v_pool, dev.ksum)
        torch.cuda.synchronize()
        outs.append({k: _host(getattr(dev, k)) for k in
                     ("h", "tau", "temp", "temp_used", "kept", "n_kept", "out", "lse", "tokens",
                      "kappa", "theta")})
    return outs


def test_checkpoint_resume_bit_identical(torch_cuda):
    from paper_2603_03310_amd.runner import Decoder
    torch = torch_cuda
    w = small(LLAMA70B_LOOP, 3, ctx=("uniform", 100, 900), steps=6, suffix="ckpt")
    x = generate(w)
    p = default_params(w).replace(rho_t=0.2, dkappa=0.1, estimator=2, est_k=64)
    fields = config_fields(w, p, x.num_pool_blocks)
    dev = upload(x)
    with Decoder(**fields) as dec:
        dec.summarize(w.batch, dev.k_pool, dev.block_tables, dev.ctx_lens, dev.ksum)
        full = _run_steps(torch, dec, dev, 0, 6)
    dev = upload(x)
    with Decoder(**fields) as dec:
        dec.summarize(w.batch, dev.k_pool, dev.block_tables, dev.ctx_lens, dev.ksum)
        first = _run_steps(torch, dec, dev, 0, 3)
        saved = {k: _host(getattr(dev, k)) for k in
                 ("h_prev", "tau", "temp", "kappa", "ctx_lens", "k_pool", "v_pool", "ksum")}
    del dev
    # Restore into fresh buffers and a fresh context.
    xr = generate(w)
    xr.h_prev, xr.tau, xr.temp = saved["h_prev"], saved["tau"], saved["temp"]
    xr.ctx_lens, xr.k_pool, xr.v_pool = saved["ctx_lens"], saved["k_pool"], saved["v_pool"]
    dev = upload(xr)
    dev.kappa.copy_(torch.from_numpy(saved["kappa"]))
    dev.ksum.copy_(torch.from_numpy(saved["ksum"]))
    with Decoder(**fields) as dec:
        rest = _run_steps(torch, dec, dev, 3, 6)
        assert dec.device_status() == 0
    for t, (a, b) in enumerate(zip(full, first + rest)):
        for k in a:
            if k == "kept":          # entries past n_kept are unspecified
                for s, n in enumerate(a["n_kept"]):
                    assert np.array_equal(a[k][s, :n], b[k][s, :n]), f"step {t}: kept of {s}"
                continue
            assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), f"step {t}: {k}"
