"""GPU parity of the calibration and safe-control guards (Section 5) through
the C ABI, against the float64 oracle: the calibration temperature wrapping
every softmax over the vocabulary, the bounded rate of change of the
temperature and of the kept fraction (with the kept-fraction state carried
on the device), and the injected entropy bias of the stress tests.  Closed
loops run several steps so the rate bounds bind; the fused step must equal
the four per-stage calls bit for bit.
"""
import math

import numpy as np
import pytest

from oracle import blocks as OB
from oracle import entropy as OE
from synth import LLAMA3_8B, LLAMA70B_LOOP, LONG_CONTEXT, TINY, default_params, generate, small
from synth.device import config_fields, upload
from tests.parity import check_step, collect, run_step
from tests.test_gpu_parity import _assert_ok, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

FIELDS = ("h", "tau", "temp", "temp_used", "row_stats", "kept", "n_kept", "scores", "theta",
          "out", "lse", "tokens", "kappa")


def _loop(torch, x, p, steps, fused=True, logit_fn=None):
    """Closed loop with the kept-fraction state; parity every step.  Returns
    the reports, the device buffers and the per-step (h, temp, kappa)."""
    from paper_2603_03310_amd.runner import Decoder
    w = x.workload
    dev = upload(x)
    reps, traj = [], []
    with Decoder(**config_fields(w, p, x.num_pool_blocks)) as dec:
        B = w.batch
        dec.summarize(B, dev.k_pool, dev.block_tables, dev.ctx_lens, dev.ksum)
        for t in range(steps):
            s_idx = min(t, x.logits.shape[0] - 1)
            if logit_fn is not None:
                dev.logits[s_idx].copy_(torch.from_numpy(logit_fn(t, x.logits[s_idx])))
            state = [a.cpu().numpy().copy() for a in (dev.h_prev, dev.tau, dev.temp, dev.kappa)]
            logits_t = dev.logits[s_idx].cpu().numpy().copy()
            run_step(dec, dev, s_idx, fused=fused, kappa=True)
            torch.cuda.synchronize()
            gpu = collect(dev, with_kappa=True)
            reps.append(check_step(k_pool=x.k_pool, v_pool=x.v_pool, tables=x.block_tables,
                                   ctx_lens=x.ctx_lens, q=x.q[s_idx], logits=logits_t,
                                   uniforms=x.uniforms[s_idx], h_prev=state[0], tau=state[1],
                                   temp=state[2], params=p, gpu=gpu, kappa=state[3]))
            traj.append((gpu.h.copy(), state[2], gpu.temp_next.copy(), state[3], gpu.kappa.copy()))
        assert dec.device_status() == 0
    return reps, dev, traj


def test_calibration_wrapper_identity(torch_cuda):
    """Logits scaled by c with T_cal = c give what the unscaled logits give
    with T_cal = 1: the same entropy, temperature update and tokens."""
    w = small(LLAMA3_8B, 4, ctx=("uniform", 100, 800), suffix="cal")
    c = 2.0
    x = generate(w)
    p1 = default_params(w)
    pc = p1.replace(t_cal=c)
    r1, d1, _ = _loop(torch_cuda, x, p1, 1)
    _assert_ok(r1)
    xs = generate(w)
    xs.logits *= np.float32(c)
    rc, dc, _ = _loop(torch_cuda, xs, pc, 1)
    _assert_ok(rc)
    assert np.max(np.abs(d1.h.cpu().numpy() - dc.h.cpu().numpy())) < 1e-4
    assert np.array_equal(d1.tokens.cpu().numpy(), dc.tokens.cpu().numpy())
    assert np.max(np.abs(d1.temp.cpu().numpy() - dc.temp.cpu().numpy())) < 1e-5


@pytest.mark.parametrize("w", [TINY, small(LLAMA3_8B, 3, ctx=("uniform", 100, 900), suffix="calp")],
                         ids=lambda w: w.name)
def test_calibration_parity(torch_cuda, w):
    p = default_params(w).replace(t_cal=0.7)
    reps, _, _ = _loop(torch_cuda, generate(w), p, 1)
    _assert_ok(reps)


def test_temperature_rate_bound_closed_loop(torch_cuda):
    """Strong gain, tight log-step bound: every step moves ln T by at most
    rho_t (inside the clip bounds), and matches the oracle."""
    w = small(LLAMA70B_LOOP, 4, ctx=("uniform", 100, 500), steps=6, suffix="rho")
    p = default_params(w).replace(eta=-0.5, rho_t=0.02)
    reps, _, traj = _loop(torch_cuda, generate(w), p, 6)
    _assert_ok(reps)
    for _, T, Tn, _, _ in traj:
        inside = (Tn > p.t_min) & (Tn < p.t_max)
        assert np.all(np.abs(np.log(Tn[inside]) - np.log(T[inside])) <= 0.02 + 1e-6)


def test_kept_fraction_rate_bound_after_entropy_collapse(torch_cuda):
    """Flat logits (entropy near log|V|: keep everything), then sharply peaked
    ones (entropy near 0): the kept fraction falls by dkappa per step, never
    faster, and the state matches the oracle every step."""
    w = small(LLAMA70B_LOOP, 4, ctx=("uniform", 300, 900), steps=5, suffix="dk")
    dk = 0.15
    p = default_params(w).replace(dkappa=dk, kappa_min=0.05)

    def logits(t, z):
        if t == 0:
            return (0.001 * z).astype(np.float32)
        out = np.full_like(z, -20.0)
        out[:, 7] = 10.0
        return out

    reps, _, traj = _loop(torch_cuda, generate(w), p, 5, logit_fn=logits)
    _assert_ok(reps)
    k0 = traj[0][4]
    assert np.all(k0 > 0.99)
    prev = k0
    for t in range(1, 5):
        cur = traj[t][4]
        assert np.all(cur >= prev - np.float32(dk) - 1e-7)
        floor = np.array([OB.kept_fraction(float(h), p) for h in traj[t][0]], dtype=np.float32)
        assert np.all(cur == np.maximum(floor, (prev - np.float32(dk)).astype(np.float32)))
        prev = cur


@pytest.mark.parametrize("bias", [-1.5, 1.0])
def test_entropy_bias(torch_cuda, bias):
    w = small(LLAMA3_8B, 4, ctx=("uniform", 100, 900), suffix=f"bias{bias}")
    p = default_params(w).replace(h_bias=bias)
    reps, dev, _ = _loop(torch_cuda, generate(w), p, 1)
    _assert_ok(reps)


@pytest.mark.parametrize("w", [
    small(LLAMA70B_LOOP, 3, ctx=("uniform", 100, 600), steps=3, suffix="guards_fused"),
    # block tables over 1024 blocks: the long-table selection
    small(LONG_CONTEXT, 2, ctx=("uniform", 9000, 17000), steps=1, suffix="guards_long"),
], ids=lambda w: w.name)
def test_fused_equals_staged_with_every_guard(torch_cuda, w):
    p = default_params(w).replace(t_cal=1.3, rho_t=0.05, dkappa=0.1, h_bias=-0.4, eta=-0.2,
                                  estimator=OE.TAIL, est_k=128, eps_h=0.1)
    steps = w.steps
    rf, df, _ = _loop(torch_cuda, generate(w), p, steps, fused=True)
    _assert_ok(rf)
    rs, ds, _ = _loop(torch_cuda, generate(w), p, steps, fused=False)
    _assert_ok(rs)
    for name in FIELDS:
        a, b = getattr(df, name).cpu().numpy(), getattr(ds, name).cpu().numpy()
        assert np.array_equal(a, b, equal_nan=True), name
