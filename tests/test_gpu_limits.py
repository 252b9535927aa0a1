"""GPU parity at the configuration limits the C ABI accepts, through the
fused step and the per-stage calls, against the float64 oracle (Sections 2-3):

* the widest block table, 16384 blocks: one sequence filling it (262144
  tokens; the selection holds 16384 keys and their encoded blocks in LDS,
  128 KB) beside a short one;
* the most query heads, H_q = 128, as G = 16 (8 KV heads) and as the widest
  KV row, H_kv * d = 2048 (16 KV heads of 128 dims, G = 8), at contexts that
  take both the one-launch selection and the long-table form.
"""
import pytest

from synth import LLAMA3_8B, LONG_CONTEXT, default_params, generate, small
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
