"""Fidelity of the mean-key block scores against the exact token-level ones.

Section 3.2 defines a block's score with the attention weights of its
tokens.  The default scoring reads one mean key per block and KV head; the
exact mode reads every key.  On the same inputs, state and entropy (hence
the same budget k), both selections run on the GPU through the C ABI, and
per workload this reports the Jaccard overlap of the two kept sets per
sequence (mean, smallest, share of identical sets), the kept fraction, and
for the long-context workload the recall of the planted high-similarity run
(the share of its full blocks each mode keeps).  The 70B-shaped loop is
measured at its first step and after the controller has settled
(--loop-step), the loop run with the mean-key scores.

    python -m paper_2603_03310_amd.fidelity [--workloads a,b,...] [--loop-step 31]

Prints one JSON line per workload (and loop step).  Parity of both scoring
modes against the float64 oracle is the GPU test suite's; nothing here reads
the oracle.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

DEFAULT = "llama3_8b_decode,long_context,skewed_mixed,llama70b_closed_loop"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workloads", default=DEFAULT)
    ap.add_argument("--loop-step", type=int, default=31)
    return ap.parse_args()


def _jaccard(a, b):
    a, b = set(a), set(b)
    return 1.0 if not a and not b else len(a & b) / len(a | b)


def compare(w, x, d, dec_mk, dec_ex, t, torch, ent):
    """Both selections on the current device state (step t's query and the
    entropy the mean-key step just produced)."""
    import numpy as np
    B = w.batch
    kept_ex = torch.full_like(d.kept, -1)
    nk_ex = torch.zeros_like(d.n_kept)
    ent.ent_block_select(dec_ex.ctx, B, d.q[t], None, d.block_tables, d.ctx_lens, d.h, kept_ex,
                         nk_ex, None, None, None, None, d.k_pool)
    torch.cuda.synchronize()
    assert dec_ex.device_status() == 0
    km, nm = d.kept.cpu().numpy(), d.n_kept.cpu().numpy()
    ke, ne = kept_ex.cpu().numpy(), nk_ex.cpu().numpy()
    ctx = d.ctx_lens.cpu().numpy()
    jac, same, frac_mk, frac_ex = [], 0, [], []
    rec_mk, rec_ex = [], []
    for s in range(B):
        a, b = km[s, :nm[s]].tolist(), ke[s, :ne[s]].tolist()
        j = _jaccard(a, b)
        jac.append(j)
        same += int(sorted(a) == sorted(b))
        nb = -(-int(ctx[s]) // 16)
        if nb:
            frac_mk.append(len(a) / nb)
            frac_ex.append(len(b) / nb)
        if x.planted is not None and x.planted[s] >= 0 and t == 0:
            off = int(x.planted[s])
            full = set(range(-(-off // 16), (off + w.planted_run) // 16))
            if full:
                rec_mk.append(len(full & set(a)) / len(full))
                rec_ex.append(len(full & set(b)) / len(full))
    out = {"workload": w.name, "loop_step": t if w.steps > 1 else None, "batch": B,
           "jaccard_mean": round(float(np.mean(jac)), 4), "jaccard_min": round(float(np.min(jac)), 4),
           "identical_sets": same,
           "kept_fraction_meankey": round(float(np.mean(frac_mk)), 4),
           "kept_fraction_exact": round(float(np.mean(frac_ex)), 4)}
    if rec_mk:
        out["planted_recall_meankey"] = round(float(np.mean(rec_mk)), 4)
        out["planted_recall_exact"] = round(float(np.mean(rec_ex)), 4)
    return out


def main():
    args = parse()
    import torch

    from paper_2603_03310_amd import ent
    from paper_2603_03310_amd.runner import Decoder
    from synth import WORKLOADS, default_params, generate
    from synth.device import config_fields, upload

    ent.load()
    torch.cuda.set_device(0)
    for name in args.workloads.split(","):
        w = WORKLOADS[name]
        x = generate(w)
        p = default_params(w)
        d = upload(x)
        fields = config_fields(w, p, x.num_pool_blocks)
        with Decoder(**fields) as dec_mk, Decoder(**dict(fields, scoring=1)) as dec_ex:
            B = w.batch
            dec_mk.summarize(B, d.k_pool, d.block_tables, d.ctx_lens, d.ksum)
            ld = d.logits.shape[2]
            stops = [0] + ([args.loop_step] if w.steps > 1 else [])
            for t in range(max(stops) + 1):
                if t in stops:
                    # The step's selection (mean-key), then the exact one on the
                    # same state and entropy; then the append.
                    ent.ent_decode_step(dec_mk.ctx, B, d.logits[t], ld, d.h_prev, d.tau, d.temp,
                                        d.q[t], d.k_pool, d.v_pool, d.ksum, d.block_tables,
                                        d.ctx_lens, d.uniforms[t], d.h, d.temp_used, d.kept,
                                        d.n_kept, d.out, d.tokens, d.row_stats, d.lse, None, None)
                    torch.cuda.synchronize()
                    print(json.dumps(compare(w, x, d, dec_mk, dec_ex, t, torch, ent)), flush=True)
                    if w.steps > 1:
                        ent.ent_kv_append(dec_mk.ctx, B, d.k_new[t], d.v_new[t], d.block_tables,
                                          d.ctx_lens, d.k_pool, d.v_pool, d.ksum)
                else:
                    ent.ent_decode_step_append(dec_mk.ctx, B, d.logits[t], ld, d.h_prev, d.tau,
                                               d.temp, d.q[t], d.k_pool, d.v_pool, d.ksum,
                                               d.block_tables, d.ctx_lens, d.uniforms[t],
                                               d.k_new[t], d.v_new[t], d.h, d.temp_used, d.kept,
                                               d.n_kept, d.out, d.tokens, d.row_stats, d.lse)
            torch.cuda.synchronize()
            assert dec_mk.device_status() == 0
        del d, x
        torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
