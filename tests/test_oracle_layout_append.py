"""Pins of the oracle's layout reader and its append step.

The layout reader is checked element by element against the documented
layout; appending tokens one at a time must give the same cache (and block
means) as building the longer sequence from scratch.
"""
import numpy as np

from oracle import append as Ap
from oracle import blocks as Bk
from oracle import layout as L
from synth import TINY, generate, small, LLAMA70B_LOOP


def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x8000, 0x4049, 0x7F80], dtype=np.uint16)
    v = L.to_f64(bits)
    assert v[0] == 1.0 and v[1] == -2.0 and v[2] == 0.0 and v[3] == 0.0
    assert v[4] == 3.140625 and v[5] == np.inf


def test_gather_matches_documented_layout():
    x = generate(TINY)
    bs = 16
    for s in range(x.workload.batch):
        N = int(x.ctx_lens[s])
        K, V = L.gather_sequence(x.k_pool, x.v_pool, x.block_tables[s], N, bs)
        assert K.shape == (N, 8, 64)
        for i in (0, 1, 15, 16, N - 1):
            p = x.block_tables[s, i // bs]
            for g in (0, 7):
                assert np.array_equal(K[i, g], x.k_pool[p, g, i % bs, :].astype(np.float64))
                assert np.array_equal(V[i, g], x.v_pool[p, g, :, i % bs].astype(np.float64))


def test_appends_equal_cache_built_from_scratch():
    w = small(LLAMA70B_LOOP, 2, ctx=("uniform", 30, 60), vocab=64, steps=20)
    x = generate(w)
    kp, vp = x.k_pool.copy(), x.v_pool.copy()
    bs = 16
    for s in range(2):
        N0 = int(x.ctx_lens[s])
        N = N0
        for t in range(19):
            N = Ap.append_token(kp, vp, x.block_tables[s], N, x.k_new[t, s], x.v_new[t, s], bs)
        assert N == N0 + 19
        K, V = L.gather_sequence(kp, vp, x.block_tables[s], N, bs)
        K0, V0 = L.gather_sequence(x.k_pool, x.v_pool, x.block_tables[s], N0, bs)
        assert np.array_equal(K[:N0], K0) and np.array_equal(V[:N0], V0)
        assert np.array_equal(K[N0:], L.to_f64(x.k_new[:19, s]))
        assert np.array_equal(V[N0:], L.to_f64(x.v_new[:19, s]))
        # block means of the grown cache equal those of the same tokens laid out at once
        ref = np.concatenate([K0, L.to_f64(x.k_new[:19, s])])
        assert np.array_equal(Bk.block_means(K, bs), Bk.block_means(ref, bs))
