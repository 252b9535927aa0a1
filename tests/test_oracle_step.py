"""Invariants of the oracle's whole step on the Tiny workload (Section 7:
bounded entropy and temperature; Section 2: entropic time never decreases;
Sections 3.2-3.3: the kept set honours the minimum block budget)."""
import math

import numpy as np

from oracle import step as St
from synth import TINY, default_params, generate


def test_tiny_step_invariants():
    x = generate(TINY)
    p = default_params(TINY)
    res = St.decode_step(k_pool=x.k_pool, v_pool=x.v_pool, tables=x.block_tables,
                         ctx_lens=x.ctx_lens, q=x.q[0], logits=x.logits[0], h_prev=x.h_prev,
                         tau=x.tau, temp=x.temp, uniforms=x.uniforms[0], params=p, block_size=16)
    for s, r in enumerate(res):
        assert 0.0 <= r["h"] <= math.log(TINY.vocab) + 1e-12
        assert r["tau"] >= float(x.tau[s])
        assert p.t_min <= r["temp_next"] <= p.t_max
        assert r["temp_used"] == float(x.temp[s])
        nb = -(-int(x.ctx_lens[s]) // 16)
        assert r["nb"] == nb
        assert len(r["kept"]) >= min(p.b_min, nb) and len(r["kept"]) >= r["k"]
        assert np.all(np.diff(r["kept"]) > 0)
        assert 0 <= r["token"] < TINY.vocab
        assert np.all(np.isfinite(r["o"]))
