"""The oracle still produces its committed outputs on the seeded Tiny workload."""
import json
import os

import numpy as np

from tests.golden.make_oracle_tiny import compute

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_oracle_tiny_regression():
    with open(os.path.join(HERE, "oracle_tiny.json")) as f:
        ref = json.load(f)
    got = compute()
    assert len(got) == len(ref)
    for a, b in zip(got, ref):
        assert a["kept"] == b["kept"] and a["token"] == b["token"] and a["k"] == b["k"]
        for key in ("h", "tau", "temp_next", "o_sum", "o_00"):
            assert np.isclose(a[key], b[key], rtol=1e-12, atol=1e-12)
