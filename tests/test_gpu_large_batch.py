"""Batches of more sequences than a plan workgroup has threads, against the oracle.

The decode's and the prologue's plans (prefix sums over the sequences'
units and scoring tiles) give each of 256 threads ceil(B / 256) sequences;
B = 600 short ragged sequences (three per thread, some empty or one token
long) through the fused step and the staged calls, checked on every
sequence: with short block tables (the prologue's dense grid, the
one-launch selection), and with one 33600-token sequence that widens the
tables past the one-launch width (the prologue's compact job list and its
plan, the long-table selection); and a three-step loop through
ent_decode_step_append checked against ent_decode_step + ent_kv_append bit
for bit.  Section 3.4 (the batched step).
"""
import numpy as np
import pytest

from synth import LLAMA3_8B, default_params, generate, small
from tests.test_gpu_parity import _assert_ok, _run, torch_cuda  # noqa: F401
from tests.test_gpu_step_append import FIELDS, _loop

pytestmark = pytest.mark.gpu

B = 600


def _workload(steps=1, wide=False):
    rng = np.random.default_rng(600)
    ctx = rng.integers(0, 300, B).tolist()
    ctx[:4] = [0, 1, 16, 17]
    if wide:
        ctx[300] = 33600
    return small(LLAMA3_8B, B, ctx=("fixed", ctx), vocab=5000, steps=steps,
                 suffix="b600_wide" if wide else "b600")


@pytest.mark.parametrize("wide", [False, True], ids=["short", "wide"])
@pytest.mark.parametrize("fused", [True, False], ids=["step", "staged"])
def test_batch_600(torch_cuda, fused, wide):
    w = _workload(wide=wide)
    x = generate(w)
    print(f"[batch] B={B}, blocks up to {w.max_blocks_per_seq}, fused={fused}", flush=True)
    reps, dev = _run(torch_cuda, x, default_params(w), fused=fused)
    _assert_ok(reps)


def test_batch_600_loop_step(torch_cuda):
    w = _workload(steps=3)
    p = default_params(w).replace(dkappa=0.1)
    a = _loop(torch_cuda, generate(w), p, fused=True)
    b = _loop(torch_cuda, generate(w), p, fused=False)
    for t, (oa, ob) in enumerate(zip(a, b)):
        for f in FIELDS:
            if f == "kept":
                for s, n in enumerate(oa["n_kept"]):
                    assert np.array_equal(oa[f][s, :n], ob[f][s, :n]), f"step {t}: kept of {s}"
                continue
            assert np.array_equal(oa[f].view(np.uint8), ob[f].view(np.uint8)), f"step {t}: {f}"
