"""GPU parity of the entropy-aware scheduler (Section 3.1 priority, Section 7
bounded priority and no starvation) through the C ABI, against the oracle's
float32 evaluation in the same operation order: selections, ages and counts
bit-exact, running means, last entropic times and priorities bit-exact as
well (the selection is an integer decided by those floats).  Several calls
in a row carry the state on the device; pools span one run of 64 indices, a
ragged tail, ties and the largest pool.
"""
import numpy as np
import pytest

from oracle import schedule as Sc
from tests.test_gpu_parity import torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

PRM = dict(alpha=1.0, beta=0.25, gamma=4.0, slo=16.0, slack_floor=0.5, gain_floor=1e-3,
           ewma_rate=0.25)


def _params(**kw):
    from types import SimpleNamespace
    from paper_2603_03310_amd import ent
    d = {**PRM, **kw}
    return ent.ent_sched_params(**d), SimpleNamespace(**d)


def _pool(rng, n, ties):
    """Seeded synthetic pool: entropic times, kept and held blocks.  With
    ties, costs and drops take few distinct values so priorities collide."""
    if ties:
        ctx = rng.choice([160, 320], size=n).astype(np.int32)
        kept = rng.choice([4, 8], size=n).astype(np.int32)
        tau = rng.choice([0.0, 1.0], size=n).astype(np.float32)
    else:
        ctx = rng.integers(0, 32768, size=n).astype(np.int32)
        kept = rng.integers(0, 512, size=n).astype(np.int32)
        tau = (rng.random(n) * 50).astype(np.float32)
    return tau, kept, ctx


def _run(torch, n, b_sels, ties, seed, prm_kw=None):
    from paper_2603_03310_amd.runner import Decoder
    from synth import LLAMA3_8B, default_params, small
    from synth.device import config_fields
    rng = np.random.default_rng(seed)
    cp, op = _params(**(prm_kw or {}))
    tau, kept, ctx = _pool(rng, n, ties)
    tau_last = tau.copy()
    gain = np.zeros(n, np.float32)
    age = np.zeros(n, np.int32)
    if not ties:
        age = rng.integers(0, 40, size=n).astype(np.int32)
        gain = (rng.random(n) * 0.5).astype(np.float32)
    cuda = "cuda:0"
    d_tau = torch.from_numpy(tau).to(cuda)
    d_kept = torch.from_numpy(kept).to(cuda)
    d_ctx = torch.from_numpy(ctx).to(cuda)
    d_tl = torch.from_numpy(tau_last).to(cuda)
    d_gain = torch.from_numpy(gain).to(cuda)
    d_age = torch.from_numpy(age).to(cuda)
    d_sel = torch.full((n,), -7, dtype=torch.int32, device=cuda)
    d_nsel = torch.full((1,), -7, dtype=torch.int32, device=cuda)
    d_pri = torch.zeros(n, dtype=torch.float32, device=cuda)
    w = small(LLAMA3_8B, 1, ctx=("uniform", 16, 32), suffix="sched")
    with Decoder(**config_fields(w, default_params(w), 4)) as dec:
        for call, b_sel in enumerate(b_sels):
            sel_o, pri_o, tl_o, g_o, age_o = Sc.schedule(tau, tau_last, gain, age, kept, ctx,
                                                         b_sel, op)
            d_sel.fill_(-7)
            dec.schedule(n, cp, d_tau, d_kept, d_ctx, d_tl, d_gain, d_age, b_sel, d_sel, d_nsel,
                         d_pri)
            torch.cuda.synchronize()
            m = int(d_nsel.item())
            tag = f"n={n} call={call} b_sel={b_sel}"
            assert m == len(sel_o), tag
            sel_g = d_sel.cpu().numpy()
            np.testing.assert_array_equal(sel_g[:m], sel_o, err_msg=tag)
            assert (sel_g[m:] == -7).all(), tag + ": wrote past n_selected"
            np.testing.assert_array_equal(d_age.cpu().numpy(), age_o, err_msg=tag)
            for name, gpu, ref in (("priority", d_pri, pri_o), ("gain", d_gain, g_o),
                                   ("tau_last", d_tl, tl_o)):
                got = gpu.cpu().numpy()
                assert np.array_equal(got.view(np.uint32), ref.astype(np.float32).view(np.uint32)), \
                    f"{tag}: {name} differs at {np.flatnonzero(got != ref)[:8]}"
            tau_last, gain, age = tl_o, g_o, age_o
            # The selected sequences run one step: their entropic time grows
            # by a drop and their kept blocks and lengths change.
            run = np.zeros(n, bool)
            run[sel_o] = True
            drop = (rng.choice([0.0, 0.5], size=n) if ties else rng.random(n) * 0.3).astype(np.float32)
            tau = np.where(run, tau + drop, tau).astype(np.float32)
            ctx = np.where(run, ctx + 1, ctx).astype(np.int32)
            if not ties:
                kept = np.where(run, rng.integers(0, 512, size=n), kept).astype(np.int32)
            d_tau.copy_(torch.from_numpy(tau))
            d_ctx.copy_(torch.from_numpy(ctx))
            d_kept.copy_(torch.from_numpy(kept))
        assert dec.device_status() == 0


@pytest.mark.parametrize("n", [1, 5, 63, 64, 65, 1000, 4099])
def test_schedule_random(torch_cuda, n):
    b = [max(1, n // 3), 0, n, n + 5, 1, max(1, n // 2), -1, max(1, n // 7)]
    _run(torch_cuda, n, b, ties=False, seed=100 + n)


@pytest.mark.parametrize("n", [7, 130, 2048])
def test_schedule_ties(torch_cuda, n):
    """Few distinct priorities: the selection must break ties by index."""
    b = [n // 2, n // 3 + 1, n - 1, 1, n // 5 + 2, n // 2]
    _run(torch_cuda, n, b, ties=True, seed=7 * n)


def test_schedule_max_pool(torch_cuda):
    from paper_2603_03310_amd import ent
    n = ent.ENT_SCHED_MAX_POOL
    _run(torch_cuda, n, [256, 256, 1024, 64, 8191], ties=False, seed=3)


def test_schedule_floors_and_weights(torch_cuda):
    """Zero cost weights but gamma, full ewma weight, a negative service
    objective (every slack at the floor)."""
    _run(torch_cuda, 300, [50, 50, 50], ties=False, seed=11,
         prm_kw=dict(alpha=0.0, beta=0.0, ewma_rate=1.0, slo=-5.0))
    _run(torch_cuda, 300, [17, 90, 3], ties=True, seed=12, prm_kw=dict(ewma_rate=0.0, gamma=0.0))


def test_schedule_serves_every_sequence(torch_cuda):
    """Section 7's no-starvation property on the device: 64 sequences with
    fixed, very unequal costs, 8 served per call, each run's entropy drop
    shrinking by 5%.  Every call matches the oracle; every sequence is
    served, the most expensive one once the cheap ones resolve."""
    from paper_2603_03310_amd.runner import Decoder
    from synth import LLAMA3_8B, default_params, small
    from synth.device import config_fields
    torch = torch_cuda
    rng = np.random.default_rng(7)
    n, b = 64, 8
    cp, op = _params(slo=24.0)
    kept = rng.integers(10, 2000, n).astype(np.int32)
    ctx = rng.integers(100, 60000, n).astype(np.int32)
    d0 = rng.uniform(0.05, 0.6, n)
    runs = np.zeros(n, dtype=np.int64)
    tau = np.zeros(n, dtype=np.float32)
    tau_last = np.zeros(n, dtype=np.float32)
    gain = np.full(n, 1.0, dtype=np.float32)
    age = np.zeros(n, dtype=np.int32)
    dv = {k: torch.from_numpy(v.copy()).to("cuda:0") for k, v in dict(
        tau=tau, kept=kept, ctx=ctx, tl=tau_last, gain=gain, age=age).items()}
    sel = torch.zeros(n, dtype=torch.int32, device="cuda:0")
    nsel = torch.zeros(1, dtype=torch.int32, device="cuda:0")
    first = np.full(n, -1)
    w = small(LLAMA3_8B, 1, ctx=("uniform", 16, 32), suffix="sched")
    with Decoder(**config_fields(w, default_params(w), 4)) as dec:
        for step in range(600):
            sel_o, _, tau_last, gain, age = Sc.schedule(tau, tau_last, gain, age, kept, ctx, b, op)
            dec.schedule(n, cp, dv["tau"], dv["kept"], dv["ctx"], dv["tl"], dv["gain"], dv["age"],
                         b, sel, nsel)
            s = sel[:b].cpu().numpy()
            np.testing.assert_array_equal(s, sel_o, err_msg=f"call {step}")
            for i in s:
                if first[i] < 0:
                    first[i] = step
                tau[i] += np.float32(d0[i] * 0.95 ** runs[i])
                runs[i] += 1
            dv["tau"].copy_(torch.from_numpy(tau))
        np.testing.assert_array_equal(dv["age"].cpu().numpy(), age)
        np.testing.assert_array_equal(dv["gain"].cpu().numpy().view(np.uint32), gain.view(np.uint32))
    assert np.all(first >= 0), np.nonzero(first < 0)[0]
    costly = int(np.argmax(1.0 * kept + 0.25 * ((ctx + 15) // 16)))
    assert first[costly] > 0
