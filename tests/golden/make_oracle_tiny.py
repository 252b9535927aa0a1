"""Write oracle_tiny.json: the oracle's outputs on the seeded Tiny workload.

Calls only the oracle and the seeded input generators."""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import step as St  # noqa: E402
from synth import TINY, default_params, generate  # noqa: E402


def compute():
    x = generate(TINY)
    p = default_params(TINY)
    res = St.decode_step(k_pool=x.k_pool, v_pool=x.v_pool, tables=x.block_tables,
                         ctx_lens=x.ctx_lens, q=x.q[0], logits=x.logits[0], h_prev=x.h_prev,
                         tau=x.tau, temp=x.temp, uniforms=x.uniforms[0], params=p, block_size=16)
    return [{"h": r["h"], "tau": r["tau"], "temp_next": r["temp_next"], "k": r["k"],
             "kept": [int(b) for b in r["kept"]], "token": r["token"],
             "o_sum": float(r["o"].sum()), "o_00": float(r["o"][0, 0])} for r in res]


if __name__ == "__main__":
    with open(os.path.join(HERE, "oracle_tiny.json"), "w") as f:
        json.dump(compute(), f, indent=1)
