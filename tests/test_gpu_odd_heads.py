"""Head layouts off the common shapes, against the oracle (Section 3.2 scoring
and selection, Section 3.4 decode).

Query-head counts whose H_q / 4 is not a power of two (the block scores
then give one lane all of a block's heads), odd KV-head counts, GQA groups
of 1 and 16, and head_dim 64, with block tables short enough for the one-launch
selection and too wide for it (the tile launch that merges L_h per tile of
256 blocks): 2500 blocks exceed the one-launch table width, and
H_q x blocks above 32768 its register budget.  With H_q = 12 and 48 the
merge of L_h runs over 42 and 10 partials per head (512 virtual threads),
not a power of two, and the sequences have more tiles than that.  Fused
step and staged calls.
"""
import pytest

from synth import LLAMA3_8B, TINY, default_params, generate, small
from tests.test_gpu_parity import _assert_ok, _run, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

# (name, KV heads, group, context lengths, head_dim)
CASES = [
    ("hq12_short", 3, 4, [1, 17, 300, 900], 128),
    ("hq12_mid", 3, 4, [1, 17, 300, 20000], 128),
    ("hq12_long", 3, 4, [1, 17, 300, 40000], 128),
    ("hq48_short", 6, 8, [5, 64, 700, 2000], 128),
    ("hq48_long", 6, 8, [5, 64, 700, 12000], 128),
    ("hq96_long", 6, 16, [33, 1000, 6000], 128),
    ("g1_long", 8, 1, [1, 300, 40000], 128),        # one query head per KV head (bf16 MFMA)
    ("d64_long", 8, 2, [7, 300, 40000], 64),        # head_dim 64 on the long-table path
]


@pytest.mark.parametrize("fused", [True, False], ids=["step", "staged"])
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_odd_head_layouts(torch_cuda, case, fused):
    name, hkv, group, ctx, hd = case
    w = small(LLAMA3_8B.replace(num_q_heads=hkv * group, num_kv_heads=hkv, head_dim=hd), len(ctx),
              ctx=("fixed", ctx), vocab=20000, suffix=name)
    print(f"[heads] {name}: H_q={hkv * group}, H_kv={hkv}, blocks up to {w.max_blocks_per_seq}",
          flush=True)
    x = generate(w)
    reps, dev = _run(torch_cuda, x, default_params(w), fused=fused)
    _assert_ok(reps)


@pytest.mark.parametrize("fused", [True, False], ids=["step", "staged"])
def test_fp32_wide_tables(torch_cuda, fused):
    """fp32 caches (block scores on the VALU) with a table too wide for the
    one-launch selection (2500 blocks): the tile launch and the merge
    launch's sampling on that path."""
    w = small(TINY, 3, ctx=("fixed", [7, 300, 40000]), suffix="f32_wide")
    x = generate(w)
    print(f"[heads] fp32 wide: blocks up to {w.max_blocks_per_seq}", flush=True)
    reps, dev = _run(torch_cuda, x, default_params(w), fused=fused)
    _assert_ok(reps)
