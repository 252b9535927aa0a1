"""ent_decode_step_append (one closed-loop step: the decode step, then the
append of the step's new token, the append sharing the step's last launch)
against ent_decode_step followed by ent_kv_append, through the C ABI: every
output, the controller and kept-fraction state, the caches, the block
summaries and the lengths agree bit for bit over a multi-step loop; bf16
batches in both selection forms (one launch per sequence, and the
long-table form: the tile launch with each sequence's selection on its last
workgroup, sampling in the last launch beside the appends) and the fp32
(VALU) path with short and wide tables.  Parity of the loop itself against the oracle:
tests/test_gpu_full_loop.py."""
import numpy as np
import pytest

from synth import LLAMA70B_LOOP, TINY, default_params, generate, small
from synth.device import config_fields, upload
from tests.test_gpu_parity import torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

CASES = [
    small(LLAMA70B_LOOP, 4, ctx=("uniform", 100, 600), steps=6, suffix="sa_one"),
    small(LLAMA70B_LOOP, 3, ctx=("uniform", 6000, 9000), steps=6, suffix="sa_three"),
    small(TINY, TINY.batch, steps=6, suffix="sa_f32"),
    small(TINY, 2, ctx=("fixed", [300, 40000]), steps=4, suffix="sa_f32_wide"),
]
FIELDS = ("h", "tau", "temp", "temp_used", "row_stats", "kept", "n_kept", "scores", "theta", "out",
          "lse", "tokens", "kappa", "ctx_lens", "k_pool", "v_pool", "ksum")


def _host(t):
    import torch
    if t.dtype == torch.bfloat16:
        t = t.view(torch.int16)
    return t.cpu().numpy().copy()


def _loop(torch, x, p, fused):
    from paper_2603_03310_amd import ent
    from paper_2603_03310_amd.runner import Decoder
    w = x.workload
    d = upload(x)
    outs = []
    with Decoder(**config_fields(w, p, x.num_pool_blocks)) as dec:
        B = w.batch
        dec.summarize(B, d.k_pool, d.block_tables, d.ctx_lens, d.ksum)
        ld = d.logits.shape[2]
        for t in range(w.steps):
            if fused:
                ent.ent_decode_step_append(dec.ctx, B, d.logits[t], ld, d.h_prev, d.tau, d.temp,
                                           d.q[t], d.k_pool, d.v_pool, d.ksum, d.block_tables,
                                           d.ctx_lens, d.uniforms[t], d.k_new[t], d.v_new[t], d.h,
                                           d.temp_used, d.kept, d.n_kept, d.out, d.tokens,
                                           d.row_stats, d.lse, d.scores, d.theta, None, d.kappa)
            else:
                ent.ent_decode_step(dec.ctx, B, d.logits[t], ld, d.h_prev, d.tau, d.temp, d.q[t],
                                    d.k_pool, d.v_pool, d.ksum, d.block_tables, d.ctx_lens,
                                    d.uniforms[t], d.h, d.temp_used, d.kept, d.n_kept, d.out,
                                    d.tokens, d.row_stats, d.lse, d.scores, d.theta, None, d.kappa)
                ent.ent_kv_append(dec.ctx, B, d.k_new[t], d.v_new[t], d.block_tables, d.ctx_lens,
                                  d.k_pool, d.v_pool, d.ksum)
            torch.cuda.synchronize()
            o = {}
            for f in FIELDS:
                src = {"temp": d.temp, "ctx_lens": d.ctx_lens, "k_pool": d.k_pool,
                       "v_pool": d.v_pool}.get(f, getattr(d, f))
                o[f] = _host(src)
            outs.append(o)
        assert dec.device_status() == 0
    return outs


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_step_append_equals_step_then_append(torch_cuda, w):
    torch = torch_cuda
    p = default_params(w).replace(dkappa=0.1)
    x = generate(w)
    a = _loop(torch, x, p, fused=True)
    b = _loop(torch, generate(w), p, fused=False)
    for t, (oa, ob) in enumerate(zip(a, b)):
        for f in FIELDS:
            if f == "kept":              # entries past n_kept are unspecified
                for s, n in enumerate(oa["n_kept"]):
                    assert np.array_equal(oa[f][s, :n], ob[f][s, :n]), f"step {t}: kept of {s}"
                continue
            assert np.array_equal(oa[f].view(np.uint8), ob[f].view(np.uint8)), f"step {t}: {f}"
    assert list(a[-1]["ctx_lens"]) == list(x.ctx_lens + w.steps)
