"""Argument checks of the entry points on a real context (they need a
device for ent_init): a bad argument returns ENT_E_INVAL with nothing
launched (the outputs keep their sentinel values) and a message; an empty
batch (B = 0) launches nothing in every entry point that takes a batch; the
exact scoring mode runs without block summaries, in the step and in append.
"""
import numpy as np
import pytest

from synth import LLAMA3_8B, default_params, generate, small
from synth.device import config_fields, upload
from tests.parity import check_step, collect, run_step
from tests.test_gpu_parity import _assert_ok, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu


def _dec(x, p):
    from paper_2603_03310_amd.runner import Decoder
    return Decoder(**config_fields(x.workload, p, x.num_pool_blocks))


def test_schedule_rejects_bad_arguments(torch_cuda):
    from paper_2603_03310_amd import ent
    torch = torch_cuda
    w = small(LLAMA3_8B, 1, ctx=("uniform", 16, 32), suffix="err")
    x = generate(w)
    n = 8
    f = lambda v: torch.full((n,), v, dtype=torch.float32, device="cuda:0")
    i = lambda v: torch.full((n,), v, dtype=torch.int32, device="cuda:0")
    sel, nsel = i(-7), i(-7)
    good = dict(alpha=1.0, beta=0.25, gamma=4.0, slo=16.0, slack_floor=0.5, gain_floor=1e-3,
                ewma_rate=0.25)
    with _dec(x, default_params(w)) as dec:
        for bad in (dict(alpha=-1.0), dict(gamma=float("inf")), dict(slack_floor=0.0),
                    dict(gain_floor=0.0), dict(ewma_rate=1.5), dict(slo=float("nan"))):
            prm = ent.ent_sched_params(**{**good, **bad})
            with pytest.raises(ent.EntError) as e:
                dec.schedule(n, prm, f(0.0), i(1), i(16), f(0.0), f(0.0), i(0), 2, sel, nsel)
            assert e.value.code == ent.ENT_E_INVAL, bad
        prm = ent.ent_sched_params(**good)
        with pytest.raises(ent.EntError) as e:
            dec.schedule(ent.ENT_SCHED_MAX_POOL + 1, prm, f(0.0), i(1), i(16), f(0.0), f(0.0),
                         i(0), 2, sel, nsel)
        assert "N must be" in str(e.value)
        with pytest.raises(ent.EntError):
            dec.schedule(n, prm, None, i(1), i(16), f(0.0), f(0.0), i(0), 2, sel, nsel)
        torch.cuda.synchronize()
        assert (sel.cpu().numpy() == -7).all() and int(nsel[0]) == -7
        dec.schedule(0, prm, None, None, None, None, None, None, 2, None, None)   # N = 0: no-op


def test_block_select_needs_the_mode_s_operand(torch_cuda):
    from paper_2603_03310_amd import ent
    w = small(LLAMA3_8B, 2, ctx=("uniform", 100, 300), suffix="err2")
    x = generate(w)
    dev = upload(x)
    for mode, missing in ((0, "ksum"), (1, "k_cache")):
        p = default_params(w).replace(scoring=mode)
        with _dec(x, p) as dec:
            kw = dict(ksum=None if mode == 0 else dev.ksum, k_cache=None if mode == 1 else dev.k_pool)
            dev.n_kept.fill_(-3)
            with pytest.raises(ent.EntError) as e:
                ent.ent_block_select(dec.ctx, 2, dev.q[0], kw["ksum"], dev.block_tables,
                                     dev.ctx_lens, dev.h, dev.kept, dev.n_kept,
                                     k_cache=kw["k_cache"])
            assert missing in str(e.value)
            assert (dev.n_kept.cpu().numpy() == -3).all()


def test_exact_step_and_append_without_summaries(torch_cuda):
    """The exact mode reads no summaries: ksum NULL in the step and in
    append; parity against the oracle after an append."""
    from oracle import append as OAp
    from paper_2603_03310_amd import ent
    torch = torch_cuda
    w = small(LLAMA3_8B, 3, ctx=("uniform", 40, 300), steps=2, suffix="nosum")
    x = generate(w)
    p = default_params(w).replace(scoring=1)
    dev = upload(x)
    kp, vp, ctx = x.k_pool.copy(), x.v_pool.copy(), x.ctx_lens.copy()
    with _dec(x, p) as dec:
        B = w.batch
        for t in range(2):
            state = [a.cpu().numpy().copy() for a in (dev.h_prev, dev.tau, dev.temp)]
            ent.ent_decode_step(dec.ctx, B, dev.logits[t], dev.logits[t].stride(0), dev.h_prev,
                                dev.tau, dev.temp, dev.q[t], dev.k_pool, dev.v_pool, None,
                                dev.block_tables, dev.ctx_lens, dev.uniforms[t], dev.h,
                                dev.temp_used, dev.kept, dev.n_kept, dev.out, dev.tokens,
                                dev.row_stats, dev.lse, dev.scores, dev.theta)
            torch.cuda.synchronize()
            rep = check_step(k_pool=kp, v_pool=vp, tables=x.block_tables, ctx_lens=ctx,
                             q=x.q[t], logits=x.logits[t], uniforms=x.uniforms[t],
                             h_prev=state[0], tau=state[1], temp=state[2], params=p,
                             gpu=collect(dev), check_ksum=False)
            _assert_ok([rep])
            ent.ent_kv_append(dec.ctx, B, dev.k_new[t], dev.v_new[t], dev.block_tables,
                              dev.ctx_lens, dev.k_pool, dev.v_pool, None)
            for s in range(B):
                ctx[s] = OAp.append_token(kp, vp, x.block_tables[s], int(ctx[s]), x.k_new[t, s],
                                          x.v_new[t, s], 16)
        assert dec.device_status() == 0
    assert list(dev.ctx_lens.cpu().numpy()) == list(ctx)


# Every buffer an entry point could write, compared byte for byte.
MUTABLE = ("ctx_lens", "k_pool", "v_pool", "h_prev", "tau", "temp", "ksum", "h", "temp_used",
           "row_stats", "kept", "n_kept", "scores", "theta", "out", "lse", "tokens", "kappa")


def _batch_calls(ent, dec, d):
    """Every entry point that takes a batch, as f(B, nul), with step 0's
    inputs; nul passes NULL for every pointer."""
    ld = d.logits[0].stride(0)

    def p(v, nul):
        return None if nul else v

    return {
        "ent_entropy_temperature": lambda B, n: ent.ent_entropy_temperature(
            dec.ctx, B, p(d.logits[0], n), ld, p(d.h_prev, n), p(d.tau, n), p(d.temp, n),
            p(d.h, n), p(d.temp_used, n), p(d.row_stats, n)),
        "ent_entropy_temperature_noalloc": lambda B, n: ent.ent_entropy_temperature_noalloc(
            dec.cfg, B, p(d.logits[0], n), ld, p(d.h_prev, n), p(d.tau, n), p(d.temp, n),
            p(d.h, n), p(d.temp_used, n), p(d.row_stats, n)),
        "ent_block_summary": lambda B, n: ent.ent_block_summary(
            dec.ctx, B, p(d.k_pool, n), p(d.block_tables, n), p(d.ctx_lens, n), p(d.ksum, n)),
        "ent_block_select": lambda B, n: ent.ent_block_select(
            dec.ctx, B, p(d.q[0], n), p(d.ksum, n), p(d.block_tables, n), p(d.ctx_lens, n),
            p(d.h, n), p(d.kept, n), p(d.n_kept, n), p(d.scores, n), p(d.theta, n), None,
            p(d.kappa, n), p(d.k_pool, n)),
        "ent_sparse_paged_decode": lambda B, n: ent.ent_sparse_paged_decode(
            dec.ctx, B, p(d.q[0], n), p(d.k_pool, n), p(d.v_pool, n), p(d.block_tables, n),
            p(d.ctx_lens, n), p(d.kept, n), p(d.n_kept, n), p(d.out, n), p(d.lse, n)),
        "ent_sample": lambda B, n: ent.ent_sample(
            dec.ctx, B, p(d.logits[0], n), ld, p(d.row_stats, n), p(d.temp_used, n),
            p(d.uniforms[0], n), p(d.tokens, n)),
        "ent_kv_append": lambda B, n: ent.ent_kv_append(
            dec.ctx, B, p(d.k_new[0], n), p(d.v_new[0], n), p(d.block_tables, n),
            p(d.ctx_lens, n), p(d.k_pool, n), p(d.v_pool, n), p(d.ksum, n)),
        "ent_decode_step": lambda B, n: ent.ent_decode_step(
            dec.ctx, B, p(d.logits[0], n), ld, p(d.h_prev, n), p(d.tau, n), p(d.temp, n),
            p(d.q[0], n), p(d.k_pool, n), p(d.v_pool, n), p(d.ksum, n), p(d.block_tables, n),
            p(d.ctx_lens, n), p(d.uniforms[0], n), p(d.h, n), p(d.temp_used, n), p(d.kept, n),
            p(d.n_kept, n), p(d.out, n), p(d.tokens, n), p(d.row_stats, n), p(d.lse, n),
            p(d.scores, n), p(d.theta, n), None, p(d.kappa, n)),
        "ent_decode_step_append": lambda B, n: ent.ent_decode_step_append(
            dec.ctx, B, p(d.logits[0], n), ld, p(d.h_prev, n), p(d.tau, n), p(d.temp, n),
            p(d.q[0], n), p(d.k_pool, n), p(d.v_pool, n), p(d.ksum, n), p(d.block_tables, n),
            p(d.ctx_lens, n), p(d.uniforms[0], n), p(d.k_new[0], n), p(d.v_new[0], n), p(d.h, n),
            p(d.temp_used, n), p(d.kept, n), p(d.n_kept, n), p(d.out, n), p(d.tokens, n),
            p(d.row_stats, n), p(d.lse, n), p(d.scores, n), p(d.theta, n), None, p(d.kappa, n)),
    }


def test_empty_batch_and_batch_bounds(torch_cuda):
    """B = 0 returns ENT_OK and launches nothing, with NULL pointers or with
    real buffers; B = -1 and B = max_batch + 1 return ENT_E_INVAL with the
    batch range in the message and nothing launched.  Every entry point that
    takes a batch; no buffer changes by a single byte."""
    from paper_2603_03310_amd import ent
    torch = torch_cuda
    w = small(LLAMA3_8B, 2, ctx=("uniform", 100, 300), steps=2, suffix="bounds")
    x = generate(w)
    d = upload(x)
    with _dec(x, default_params(w)) as dec:
        dec.summarize(w.batch, d.k_pool, d.block_tables, d.ctx_lens, d.ksum)
        for f in ("h", "temp_used", "row_stats", "scores", "theta", "out", "lse"):
            getattr(d, f).fill_(-5.0)
        for f in ("kept", "n_kept", "tokens"):
            getattr(d, f).fill_(-5)
        torch.cuda.synchronize()
        before = {f: getattr(d, f).clone() for f in MUTABLE}
        for name, call in _batch_calls(ent, dec, d).items():
            print(f"[bounds] {name}", flush=True)
            call(0, True)
            call(0, False)
            for B in (-1, w.batch + 1):
                with pytest.raises(ent.EntError) as e:
                    call(B, False)
                assert e.value.code == ent.ENT_E_INVAL, (name, B)
                assert "B must be in [0, max_batch]" in str(e.value), (name, B)
        torch.cuda.synchronize()
        for f in MUTABLE:
            a, b = getattr(d, f), before[f]
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f
        assert dec.device_status() == 0
