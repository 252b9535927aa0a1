"""Sampling over many logit chunks and at the uniform's extremes, against the oracle.

The sampler (Sections 2.1 and 3.3: the next token drawn at the controlled
temperature) first picks a chunk of 4096 logits from the chunk statistics
(four chunks per lane of one wave, up to 256 chunks), then the token inside
it.  Rows at |V| = 300000 (74 chunks) and |V| = 1048576 (256 chunks, the
largest vocabulary): mass only in the first chunk, only in the last chunk,
only at the very last token, two equal spikes at the two ends of the row,
and generated rows; uniforms 0, 1e-7, 0.5 and the largest float below 1.
The whole step runs fused and as staged calls, with block tables short
enough for the one-launch selection (sampling beside it) and too wide for
it (sampling in the merge launch); tokens are checked by the oracle's rule
(equal, or inside the tie band, tests/parity.py), and the forced rows by
where their mass lies.
"""
import numpy as np
import pytest

from synth import SKEWED, default_params, generate, small
from tests.test_gpu_parity import _assert_ok, _run, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

U_EDGES = np.array([0.0, 1e-7, 0.5, np.nextafter(np.float32(1.0), np.float32(0.0))],
                   dtype=np.float32)
# Context lengths: every table short enough for the one-launch selection, or
# one sequence long enough that H_q x blocks exceeds it.
CTX = {"short": [16, 100, 300, 64, 1, 33, 200, 17],
       "wide": [16, 100, 20000, 5000, 1, 33, 200, 17]}


@pytest.mark.parametrize("vocab", [300000, 1048576])
@pytest.mark.parametrize("tables", ["short", "wide"])
@pytest.mark.parametrize("fused", [True, False])
def test_sample_many_chunks_and_edge_uniforms(torch_cuda, vocab, tables, fused):
    B = 8
    w = small(SKEWED, B, ctx=("fixed", CTX[tables]), vocab=vocab, suffix=f"sample_{tables}")
    x = generate(w)
    V = vocab
    C = -(-V // 4096)
    print(f"[sample] V={V} ({C} chunks), {tables} tables, fused={fused}", flush=True)
    lg = x.logits[0]
    rng = np.random.default_rng(7)
    lg[0] = -np.inf
    lg[0, :4096] = rng.normal(0.0, 2.0, 4096)                 # first chunk only
    lg[1] = -np.inf
    lg[1, (C - 1) * 4096:] = rng.normal(0.0, 2.0, V - (C - 1) * 4096)   # last chunk only
    lg[2] = -np.inf
    lg[2, V - 1] = 3.0                                        # the very last token only
    lg[3] = -np.inf
    lg[3, [0, V - 1]] = 0.0                                   # two equal spikes at the ends
    x.uniforms[0] = np.tile(U_EDGES, 2)
    p = default_params(w)
    reps, dev = _run(torch_cuda, x, p, fused=fused)
    _assert_ok(reps)
    tok = dev.tokens.cpu().numpy()
    assert 0 <= tok[0] < 4096
    assert (C - 1) * 4096 <= tok[1] < V
    assert tok[2] == V - 1
    assert tok[3] in (0, V - 1)
    assert np.all((tok >= 0) & (tok < V))
