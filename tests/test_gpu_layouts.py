"""GPU parity of logit-row layouts and of a large attention score range,
through the C ABI, against the float64 oracle (bands in tests/parity.py).

Row layouts: the ABI accepts logit rows with a stride ld >= |V|; rows that
are not 16-byte aligned (ld % 4 != 0) or a vocabulary that is not a
multiple of the 4096-logit chunk take the kernels' scalar-load variants
(entropy chunk passes, sampling, the estimators' re-read).  Cases: a padded
buffer of width |V| + 3 viewed as [:, :|V|] with NaN in the padding (a read
past the row would poison the results), and |V| = 5001 (a ragged last chunk
with ld = |V|), each through the one-call step and the per-stage calls
(which must agree bit for bit) and through an estimator mode.

Score range: keys and values scaled by 16, and per (sequence, KV head) one
token whose key is 16 times the sum of its group's queries, so that this
token carries essentially all of every head's attention mass and the other
scores span hundreds of nats below it: the online rescaling of the decode
and the split of the probabilities into two bf16 parts see their extremes.
"""
import math

import numpy as np
import pytest

from oracle import layout as OL
from synth import LLAMA3_8B, TINY, bf16_bits_to_f32, default_params, f32_to_bf16_bits, generate, small
from synth.device import config_fields, upload
from tests.parity import check_step, collect, run_step
from tests.test_gpu_parity import torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

FIELDS = ("h", "tau", "temp", "temp_used", "row_stats", "kept", "n_kept", "scores", "theta",
          "out", "lse", "tokens")


def _pad_rows(torch, dev, pad):
    """Replace dev.logits [S, B, V] by a view of a [S, B, V + pad] buffer
    whose padding holds NaN; returns the row stride."""
    if pad == 0:
        return dev.logits.shape[-1]
    S, B, V = dev.logits.shape
    buf = torch.full((S, B, V + pad), float("nan"), dtype=torch.float32, device=dev.logits.device)
    buf[:, :, :V] = dev.logits
    dev.logits = buf[:, :, :V]
    return V + pad


def _run_layout(torch, x, p, pad, fused):
    from paper_2603_03310_amd.runner import Decoder
    w = x.workload
    dev = upload(x)
    ld = _pad_rows(torch, dev, pad)
    assert dev.logits[0].stride(0) == ld
    with Decoder(**config_fields(w, p, x.num_pool_blocks)) as dec:
        dec.summarize(w.batch, dev.k_pool, dev.block_tables, dev.ctx_lens, dev.ksum)
        state = (x.h_prev.copy(), x.tau.copy(), x.temp.copy())
        run_step(dec, dev, 0, fused=fused)
        torch.cuda.synchronize()
        assert dec.device_status() == 0
    gpu = collect(dev)
    rep = check_step(k_pool=x.k_pool, v_pool=x.v_pool, tables=x.block_tables, ctx_lens=x.ctx_lens,
                     q=x.q[0], logits=x.logits[0], uniforms=x.uniforms[0], h_prev=state[0],
                     tau=state[1], temp=state[2], params=p, gpu=gpu)
    assert rep.ok(), "; ".join(rep.failures[:8])
    assert np.all(np.isfinite(gpu.h)) and np.all(np.isfinite(gpu.out))
    print(f"[layout] {w.name} ld={ld} fused={fused}: entropy err {rep.max_h_err:.2e}, "
          f"attention err {rep.max_att_err:.2e}", flush=True)
    return dev


LAYOUT_CASES = [
    ("tiny_pad3", TINY, 3),
    ("l8_pad3", small(LLAMA3_8B, 4, ctx=("uniform", 100, 1500), suffix="pad3"), 3),
    ("l8_v5001", small(LLAMA3_8B, 4, ctx=("uniform", 100, 1500), vocab=5001, suffix="v5001"), 0),
    ("tiny_v5001_pad3", small(TINY, 4, vocab=5001, suffix="v5001"), 3),
]


@pytest.mark.parametrize("name,w,pad", LAYOUT_CASES, ids=[c[0] for c in LAYOUT_CASES])
def test_row_layouts_fused_and_staged(torch_cuda, name, w, pad):
    """Unaligned and ragged logit rows: parity of the one-call step and of the
    per-stage calls, which agree bit for bit."""
    torch = torch_cuda
    p = default_params(w)
    x = generate(w)
    df = _run_layout(torch, x, p, pad, fused=True)
    ds = _run_layout(torch, generate(w), p, pad, fused=False)
    for f in FIELDS:
        a, b = getattr(df, f).cpu().numpy(), getattr(ds, f).cpu().numpy()
        assert np.array_equal(a, b, equal_nan=True), f


@pytest.mark.parametrize("est", [1, 2], ids=["topk", "tail"])
@pytest.mark.parametrize("name,w,pad", LAYOUT_CASES[1:3], ids=[c[0] for c in LAYOUT_CASES[1:3]])
def test_row_layouts_estimators(torch_cuda, name, w, pad, est):
    """The estimators re-read the logits of the top threads (scalar loads on
    these rows): parity of the estimate, the controller and the guarded
    budget acting on it, fused and staged alike."""
    torch = torch_cuda
    p = default_params(w).replace(estimator=est, est_k=64, eps_h=0.25)
    df = _run_layout(torch, generate(w), p, pad, fused=True)
    ds = _run_layout(torch, generate(w), p, pad, fused=False)
    for f in FIELDS:
        a, b = getattr(df, f).cpu().numpy(), getattr(ds, f).cpu().numpy()
        assert np.array_equal(a, b, equal_nan=True), f


def _scale_bits(bits, c):
    """bf16 bits times an exact power of two c."""
    return f32_to_bf16_bits(bf16_bits_to_f32(bits) * np.float32(c))


def _large_range_inputs(w, seed_tokens=7):
    """Keys and values x16; per (sequence, KV head) one dominant token whose
    key is 16 x the sum of the group's step-0 queries.  Returns the inputs and
    the dominant token positions [B]."""
    x = generate(w)
    bf = w.kv_dtype == "bf16"
    c = 16.0
    if bf:
        x.k_pool[...] = _scale_bits(x.k_pool, c)
        x.v_pool[...] = _scale_bits(x.v_pool, c)
    else:
        x.k_pool *= np.float32(c)
        x.v_pool *= np.float32(c)
    rng = np.random.default_rng(seed_tokens)
    G, bs = w.group, w.block_size
    pos = np.zeros(w.batch, dtype=np.int64)
    for s in range(w.batch):
        N = int(x.ctx_lens[s])
        i = int(rng.integers(0, N))
        pos[s] = i
        p = int(x.block_tables[s][i // bs])
        qf = OL.to_f64(x.q[0, s])
        for g in range(w.num_kv_heads):
            key = (16.0 * qf[g * G:(g + 1) * G].sum(axis=0)).astype(np.float32)
            x.k_pool[p, g, i % bs, :] = f32_to_bf16_bits(key) if bf else key
    return x, pos


@pytest.mark.parametrize("w", [small(LLAMA3_8B, 4, ctx=("uniform", 300, 2500), suffix="range"),
                               small(TINY, 4, suffix="range")], ids=lambda w: w.name)
def test_large_score_range(torch_cuda, w):
    """One token holds >= 0.99 of every head's attention mass (checked on the
    oracle side), the rest span a wide score range: parity of attention,
    scores and kept lists, with every block kept (so the dominant token is
    attended) and with the default budget."""
    from paper_2603_03310_amd.runner import Decoder
    torch = torch_cuda
    x, pos = _large_range_inputs(w)
    # The case is what it claims: in the oracle's dense attention the
    # dominant token's weight is >= 0.99 for every head.
    for s in range(w.batch):
        K, _ = OL.gather_sequence(x.k_pool, x.v_pool, x.block_tables[s], int(x.ctx_lens[s]), 16)
        qf = OL.to_f64(x.q[0, s])
        p0 = default_params(w)
        for h in range(w.num_q_heads):
            sc = p0.scale * (K[:, h // w.group, :] @ qf[h])
            a = np.exp(sc - sc.max())
            a /= a.sum()
            assert a[pos[s]] >= 0.99, (s, h, a[pos[s]])
            assert sc.max() - np.sort(sc)[-2] > 20.0
    for kappa_min in (1.0, default_params(w).kappa_min):
        p = default_params(w).replace(kappa_min=kappa_min)
        for fused in (True, False):
            dev = upload(x)
            with Decoder(**config_fields(w, p, x.num_pool_blocks)) as dec:
                dec.summarize(w.batch, dev.k_pool, dev.block_tables, dev.ctx_lens, dev.ksum)
                run_step(dec, dev, 0, fused=fused)
                torch.cuda.synchronize()
                assert dec.device_status() == 0
            gpu = collect(dev)
            rep = check_step(k_pool=x.k_pool, v_pool=x.v_pool, tables=x.block_tables,
                             ctx_lens=x.ctx_lens, q=x.q[0], logits=x.logits[0],
                             uniforms=x.uniforms[0], h_prev=x.h_prev, tau=x.tau, temp=x.temp,
                             params=p, gpu=gpu)
            assert rep.ok(), "; ".join(rep.failures[:8])
            print(f"[range] {w.name} kappa_min={kappa_min} fused={fused}: attention err "
                  f"{rep.max_att_err:.2e}, score err {rep.max_score_err:.2e} "
                  f"(rel {rep.max_score_rel_err:.2e})", flush=True)
            if kappa_min == 1.0:
                # Keep-all: the output is the dominant token's value row.
                assert list(gpu.n_kept) == [-(-int(n) // 16) for n in x.ctx_lens]
