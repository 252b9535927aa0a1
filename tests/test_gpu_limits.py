"""GPU parity at the configuration limits the C ABI accepts, through the
fused step and the per-stage calls, against the float64 oracle (Sections 2-3):

* the widest block table, 16384 blocks: one sequence filling it (262144
  tokens; the selection holds 16384 keys and their encoded blocks in LDS,
  128 KB) beside a short one;
* the most query heads, H_q = 128, as G = 16 (8 KV heads) and as the widest
  KV row, H_kv * d = 2048 (16 KV heads of 128 dims, G = 8), at contexts that
  take both the one-launch selection and the long-table form;
* more kept units (sequence, KV head, block) in one decode than 2^31 divided
  by its ranges, so that locating the range of a unit needs 64-bit
  products: block tables that name the blocks of a small pool many times
  over, every block kept.
"""
import numpy as np
import pytest

from synth import LLAMA3_8B, LONG_CONTEXT, TINY, default_params, generate, small
from synth.gen import Inputs, f32_to_bf16_bits
from tests.test_gpu_parity import _assert_ok, _run, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

MAX_BLOCKS = 16384


@pytest.mark.parametrize("fused", [True, False], ids=["step", "staged"])
def test_widest_block_table(torch_cuda, fused):
    w = small(LONG_CONTEXT.replace(num_q_heads=8, num_kv_heads=2), 2,
              ctx=("fixed", [MAX_BLOCKS * 16, 300]), vocab=5000, suffix="max_table")
    assert w.max_blocks_per_seq == MAX_BLOCKS
    print(f"[limits] {w.name}: blocks up to {w.max_blocks_per_seq}", flush=True)
    x = generate(w)
    reps, dev = _run(torch_cuda, x, default_params(w), fused=fused)
    _assert_ok(reps)
    assert 0 < int(dev.n_kept[0]) <= MAX_BLOCKS


# (name, KV heads, group, context lengths)
HEADS = [
    ("hq128_g16_short", 8, 16, [1, 300, 2000]),
    ("hq128_g16_long", 8, 16, [1, 300, 20000]),
    ("hkv16_d128_short", 16, 8, [17, 900, 2000]),
    ("hkv16_d128_long", 16, 8, [17, 900, 20000]),
]


@pytest.mark.parametrize("fused", [True, False], ids=["step", "staged"])
@pytest.mark.parametrize("case", HEADS, ids=[c[0] for c in HEADS])
def test_most_query_heads(torch_cuda, case, fused):
    name, hkv, group, ctx = case
    w = small(LLAMA3_8B.replace(num_q_heads=hkv * group, num_kv_heads=hkv), len(ctx),
              ctx=("fixed", ctx), vocab=20000, suffix=name)
    assert w.num_q_heads == 128 and w.num_kv_heads * w.head_dim <= 2048
    print(f"[limits] {name}: H_q={w.num_q_heads}, H_kv={hkv}, blocks up to "
          f"{w.max_blocks_per_seq}", flush=True)
    x = generate(w)
    reps, dev = _run(torch_cuda, x, default_params(w), fused=fused)
    _assert_ok(reps)


def _aliased(base, batch, nb, seed):
    """`batch` sequences of nb full blocks whose tables name the blocks of
    `base`'s generated pool at random, many times over."""
    xp = generate(base)
    w = base.replace(batch=batch, ctx=("fixed", [16 * nb] * batch), name=f"{base.name}_aliased")
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((1, batch, w.num_q_heads, w.head_dim)).astype(np.float32)
    if w.kv_dtype == "bf16":
        q = f32_to_bf16_bits(q)
    return Inputs(workload=w, ctx_lens=np.full(batch, 16 * nb, np.int32),
                  block_tables=rng.integers(0, xp.num_pool_blocks, size=(batch, nb), dtype=np.int32),
                  num_pool_blocks=xp.num_pool_blocks, k_pool=xp.k_pool, v_pool=xp.v_pool, q=q,
                  logits=rng.standard_normal((1, batch, w.vocab)).astype(np.float32),
                  h_prev=rng.uniform(0.0, np.log(w.vocab), batch).astype(np.float32),
                  tau=np.zeros(batch, np.float32), temp=np.ones(batch, np.float32),
                  uniforms=rng.random((1, batch)).astype(np.float32), k_new=None, v_new=None,
                  planted=None)


# (name, workload, sequences, blocks each): 1024 x 4200 = 4300800 > 2^22 units for
# the bf16 decode's ranges per workgroup (512 of them), 512 x 4200 = 2150400 > 2^21
# for the fp32 decode's ranges per wave (1024 or more).
MANY_UNITS = [
    ("bf16_4M", small(LLAMA3_8B.replace(num_q_heads=8, num_kv_heads=1, head_dim=64), 4,
                      ctx=("fixed", [2048] * 4), vocab=1024, suffix="units"), 1024, 4200),
    ("f32_2M", small(TINY.replace(num_q_heads=8, num_kv_heads=1), 4,
                     ctx=("fixed", [2048] * 4), suffix="units"), 512, 4200),
]


@pytest.mark.parametrize("fused", [True, False], ids=["step", "staged"])
@pytest.mark.parametrize("case", MANY_UNITS, ids=[c[0] for c in MANY_UNITS])
def test_kept_units_past_32_bit_products(torch_cuda, case, fused):
    name, base, batch, nb = case
    x = _aliased(base, batch, nb, seed=11)
    w = x.workload
    # An error bound past log |V| floors the budget's entropy above it: every block is kept.
    p = default_params(w).replace(eps_h=100.0)
    print(f"[limits] {name}: {batch * nb * w.num_kv_heads} kept units", flush=True)
    reps, dev = _run(torch_cuda, x, p, seqs=[0, 1, batch - 2, batch - 1], fused=fused)
    _assert_ok(reps)
    assert (dev.n_kept.cpu().numpy() == nb).all()
