"""The 70B-shaped closed loop at full size and full length, against the oracle.

Batch 128, 64/8 heads, d = 128, contexts U[4096, 16384], |V| = 128256: all
64 steps run on the device as the benchmark runs them (ent_decode_step_append:
the decode step, then the append of its token's K/V, the controller and
kept-fraction state carried in device memory).  At steps 0, 15, 31, 47 and 63
the step is checked against the oracle on sampled sequences, teacher-forced
(tests/parity.py): the oracle reads the state the step started from, and
host copies of the pools that receive the same appended tokens.  The late
steps are the low-kept-fraction regime the controller drives these rows to
(temperatures near their equilibrium, about a tenth of the blocks kept).
"""
import numpy as np
import pytest

from oracle import append as OAp
from synth import LLAMA70B_LOOP, default_params, generate
from synth.device import config_fields, upload
from tests.parity import check_step, collect
from tests.test_gpu_parity import _sampled, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

CHECK_STEPS = (0, 15, 31, 47, 63)


def test_full_size_70b_loop_all_steps(torch_cuda):
    from paper_2603_03310_amd import ent
    from paper_2603_03310_amd.runner import Decoder
    torch = torch_cuda
    w = LLAMA70B_LOOP
    x = generate(w)
    p = default_params(w)
    seqs = _sampled(w.batch, 4, 5)
    print(f"[loop] full-size {w.name}, {w.steps} steps, sampled sequences {seqs}", flush=True)
    dev = upload(x)
    kp, vp = x.k_pool, x.v_pool          # host pools, appended in step with the device's
    ctx = x.ctx_lens.copy()
    fractions = {}
    failures = []
    with Decoder(**config_fields(w, p, x.num_pool_blocks)) as dec:
        B = w.batch
        dec.summarize(B, dev.k_pool, dev.block_tables, dev.ctx_lens, dev.ksum)
        for t in range(w.steps):
            check = t in CHECK_STEPS
            if check:
                torch.cuda.synchronize()
                state = [a.cpu().numpy().copy() for a in (dev.h_prev, dev.tau, dev.temp, dev.kappa)]
                # The summaries the step scores with (the step's append then
                # refreshes the last block's).
                ksum_pre = dev.ksum.cpu().numpy().copy()
            ent.ent_decode_step_append(dec.ctx, B, dev.logits[t], dev.logits.shape[2], dev.h_prev,
                                       dev.tau, dev.temp, dev.q[t], dev.k_pool, dev.v_pool,
                                       dev.ksum, dev.block_tables, dev.ctx_lens, dev.uniforms[t],
                                       dev.k_new[t], dev.v_new[t], dev.h, dev.temp_used, dev.kept,
                                       dev.n_kept, dev.out, dev.tokens, dev.row_stats, dev.lse,
                                       dev.scores, dev.theta, None, dev.kappa)
            if check:
                torch.cuda.synchronize()
                gpu = collect(dev, with_kappa=True)
                gpu.ksum = ksum_pre
                nb_all = sum(-(-int(n) // 16) for n in ctx)
                fractions[t] = float(gpu.n_kept.sum()) / nb_all
                rep = check_step(k_pool=kp, v_pool=vp, tables=x.block_tables, ctx_lens=ctx,
                                 q=x.q[t], logits=x.logits[t], uniforms=x.uniforms[t],
                                 h_prev=state[0], tau=state[1], temp=state[2], params=p, gpu=gpu,
                                 seqs=seqs, kappa=state[3])
                print(f"[loop] step {t}: kept fraction {fractions[t]:.4f}, mean temperature "
                      f"{float(state[2].mean()):.3f}, entropy err {rep.max_h_err:.2e}, score err "
                      f"{rep.max_score_err:.2e} (rel {rep.max_score_rel_err:.2e}), attention err "
                      f"{rep.max_att_err:.2e}, band {rep.band_exempt}", flush=True)
                failures += [f"step {t}: {m}" for m in rep.failures]
            # Only the sampled sequences' blocks are read on the host.
            for s in seqs:
                ctx[s] = OAp.append_token(kp, vp, x.block_tables[s], int(ctx[s]), x.k_new[t, s],
                                          x.v_new[t, s], 16)
            for s in set(range(B)) - set(seqs):
                ctx[s] += 1
        torch.cuda.synchronize()
        assert dec.device_status() == 0
    assert not failures, "; ".join(failures[:8])
    assert list(dev.ctx_lens.cpu().numpy()) == list(x.ctx_lens + w.steps)
    # The late steps are the pruned regime: far fewer blocks kept than at step 0.
    assert fractions[63] < 0.5 * fractions[0]
