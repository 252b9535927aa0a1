"""One closed-loop step (ent_decode_step_append, Section 3.4) captured in a
HIP graph and replayed, against the same call made eagerly, bit for bit.

The calls allocate, clear and synchronise nothing, and the counters that the
long-table form's tile launch uses to pick each sequence's selecting
workgroup return to zero by the end of every step, so a graph of the step
replays exactly.  Two block-table forms: too wide for the one-launch
selection (64 query heads, a 20000-token sequence: the tile launch with its
per-sequence counters) and short enough for it.  The state the step changes
(controller and kept-fraction state, lengths, caches, block summaries) is
restored and every output filled with a sentinel before the eager call and
before every replay; between replays the program does eager work of its
own; every replay's outputs and state equal the eager step's.
"""
import numpy as np
import pytest

from synth import LLAMA3_8B, LLAMA70B_LOOP, default_params, generate, small
from synth.device import config_fields, upload
from tests.test_gpu_parity import torch_cuda  # noqa: F401
from tests.test_gpu_step_append import FIELDS, _host

pytestmark = pytest.mark.gpu

CASES = [
    small(LLAMA70B_LOOP, 3, ctx=("fixed", [300, 20000, 9000]), steps=2, suffix="graph_wide"),
    small(LLAMA3_8B, 4, ctx=("fixed", [1, 300, 2000, 900]), steps=2, suffix="graph_short"),
]
STATE = ("h_prev", "tau", "temp", "kappa", "ctx_lens", "k_pool", "v_pool", "ksum")
OUTPUTS = ("h", "temp_used", "row_stats", "kept", "n_kept", "scores", "theta", "out", "lse",
           "tokens")
REPLAYS = 4


def _clear_outputs(torch, d):
    """The same sentinel in every output before each call, so that a replay
    that wrote nothing cannot match."""
    for f in OUTPUTS:
        t = getattr(d, f)
        t.fill_(float("nan") if t.dtype.is_floating_point else -7)


def _step(ent, dec, d, B, ld, stream):
    ent.ent_decode_step_append(dec.ctx, B, d.logits[0], ld, d.h_prev, d.tau, d.temp, d.q[0],
                               d.k_pool, d.v_pool, d.ksum, d.block_tables, d.ctx_lens,
                               d.uniforms[0], d.k_new[0], d.v_new[0], d.h, d.temp_used, d.kept,
                               d.n_kept, d.out, d.tokens, d.row_stats, d.lse, d.scores, d.theta,
                               stream, d.kappa)


def _snapshot(d):
    return {f: _host(getattr(d, f)) for f in FIELDS + ("h_prev",)}


def _same(ref, got, tag):
    for f, a in ref.items():
        b = got[f]
        if f == "kept":
            for s, n in enumerate(ref["n_kept"]):
                assert np.array_equal(a[s, :n], b[s, :n]), f"{tag}: kept of {s}"
            continue
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"{tag}: {f}"


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_step_graph_replays_equal_eager(torch_cuda, w):
    torch = torch_cuda
    from paper_2603_03310_amd import ent
    from paper_2603_03310_amd.runner import Decoder
    p = default_params(w).replace(dkappa=0.1)
    x = generate(w)
    d = upload(x)
    print(f"[graph] {w.name}: blocks up to {w.max_blocks_per_seq}", flush=True)
    with Decoder(**config_fields(w, p, x.num_pool_blocks)) as dec:
        B = w.batch
        ld = d.logits.shape[2]
        dec.summarize(B, d.k_pool, d.block_tables, d.ctx_lens, d.ksum)
        torch.cuda.synchronize()
        saved = {f: getattr(d, f).clone() for f in STATE}

        def restore():
            for f in STATE:
                getattr(d, f).copy_(saved[f])
            _clear_outputs(torch, d)
            torch.cuda.synchronize()

        restore()
        _step(ent, dec, d, B, ld, None)
        torch.cuda.synchronize()
        ref = _snapshot(d)
        restore()
        s = torch.cuda.Stream()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            _step(ent, dec, d, B, ld, s)
        for r in range(REPLAYS):
            restore()
            g.replay()
            torch.cuda.synchronize()
            _same(ref, _snapshot(d), f"replay {r}")
            # Eager work of the program's own between replays.
            assert torch.isfinite(d.out).all().item()
        assert dec.device_status() == 0
