"""Benchmark of entropic-time decode steps on one MI355X.

A step is the whole hot path over one batch: entropy and controller, block
scoring and selection, kept-block decode attention and sampling (one
ent_decode_step call), and in a closed loop the append of the new token's
K/V (ent_kv_append).  Inputs are seeded synthetic data of the named
workload, resident in HBM before timing.

Default workload: the 70B-shaped closed loop (one ent_decode_step_append call
per loop step) (batch 128, 64/8 heads, d 128,
contexts U[4096, 16384], |V| 128256, 64 loop steps with fresh logits and one
appended token per step, state on the device).  --warmup loop steps run
untimed, then --steps consecutive loop steps are timed; the roofline is the
decode entry point (attention and segment merge) replayed once per timed
step, back to back between two HIP events on the launch stream, on that
step's kept lists.

Single-step workloads (--workload llama3_8b_decode, long_context,
skewed_mixed, tiny): --steps fused steps timed back to back; --copies copies
of every input rotate between steps so the 256 MB Infinity Cache cannot
serve a step from the previous one, and every step starts from a fresh copy
of the controller state, so all timed steps do identical work; a second
pass issues the same steps through the per-stage entry points with events
between them, and a third the decode entry point alone (the roofline).

Prints one JSON line: decode steps/s, the achieved HBM rate on kept KV +
logit bytes and on every byte the step moves, the roofline of the dominant
kernel, and the float64 oracle timed on the host's cores on a bounded sample
of the same workload.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
                    [--estimator exact|topk|tail] [--est-k K] [--eps-h E]
                    [--scoring meankey|exact] [--keep-first N] [--keep-last N]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "decode steps/sec and achieved HBM GB/s (kept KV + logits) vs peak, 1 MI355X"
# Sources of the decode entry point's kernels (attention and segment merge).
DECODE_SRCS = [os.path.join(ROOT, "paper_2603_03310_amd", "csrc", f)
               for f in ("decode.hip", "ent_internal.h")]


def decode_src_digest() -> str:
    h = hashlib.sha256()
    for f in DECODE_SRCS:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=59)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama70b_closed_loop")
    ap.add_argument("--copies", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--estimator", choices=["exact", "topk", "tail"], default="exact",
                    help="entropy the controller acts on (top-k / tail-corrected estimates)")
    ap.add_argument("--est-k", type=int, default=256)
    ap.add_argument("--eps-h", type=float, default=None,
                    help="estimator error bound in the block budget (default 0)")
    ap.add_argument("--scoring", choices=["meankey", "exact"], default="meankey",
                    help="block scores from mean keys, or from exact token-level weights")
    ap.add_argument("--keep-first", type=int, default=0, help="leading blocks always kept")
    ap.add_argument("--keep-last", type=int, default=0, help="trailing blocks always kept")
    ap.add_argument("--q-heads", type=int, default=None,
                    help="query heads (the GQA group is q-heads / the workload's KV heads)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration)")
    return ap.parse_args()


def kv_bytes_kept(x, n_kept, kept, elem):
    """Bytes of K and V in the kept blocks (valid tokens only)."""
    w = x.workload
    per_tok = w.num_kv_heads * w.head_dim * 2 * elem
    tot = 0
    for s in range(w.batch):
        N = int(x.ctx_lens[s])
        nb = -(-N // 16)
        ks = kept[s][: int(n_kept[s])]
        toks = 16 * len(ks)
        if nb and (nb - 1) in set(ks.tolist()):
            toks -= 16 - (N - 16 * (nb - 1))
        tot += toks * per_tok
    return tot


def total_bytes(w, ctx_lens, kv_kept, elem, scoring):
    """Every byte the step must move (besides the metric's kept K/V and
    logits): one logit chunk re-read per row by sampling, the block
    summaries (mean-key scoring) or every valid key (exact scoring), the
    queries and the attention outputs."""
    B, V = w.batch, w.vocab
    nb = sum(-(-int(n) // 16) for n in ctx_lens)
    if scoring:
        scores = int(sum(int(n) for n in ctx_lens)) * w.num_kv_heads * w.head_dim * elem
    else:
        scores = nb * w.num_kv_heads * w.head_dim * 4
    return (4 * B * V + 4 * B * 4096 + scores + kv_kept
            + B * w.num_q_heads * w.head_dim * (elem + 4))


_BASE = None   # (inputs, params) of the CPU baseline, shared with forked workers


def _oracle_worker(args):
    """Sequence-steps of the oracle for about `seconds` (one thread); returns
    how many ran and the time.  Single-step workloads: sequences start,
    start + stride, ... of the step.  Closed loops: the same sequences, each
    run through consecutive loop steps from step 0 with the oracle's own
    controller and kept-fraction state and its own appended tokens (on the
    worker's copy-on-write view of the pools)."""
    start, stride, seconds = args
    x, p = _BASE
    from threadpoolctl import threadpool_limits

    from oracle import append as OAp
    from oracle import step as St
    B, S = x.workload.batch, x.steps
    loop = S > 1
    h_prev, tau, temp = (a.astype(np.float64).copy() for a in (x.h_prev, x.tau, x.temp))
    kappa = np.full(B, np.nan)
    ctx = x.ctx_lens.copy()
    done, s, t = 0, start % B, 0
    t0 = time.perf_counter()
    with threadpool_limits(limits=1):
        while done == 0 or time.perf_counter() - t0 < seconds:
            if loop and t == 0:       # the sequence starts the loop from its initial state
                h_prev[s], tau[s], temp[s] = x.h_prev[s], x.tau[s], x.temp[s]
                kappa[s], ctx[s] = np.nan, x.ctx_lens[s]
            o = St.sequence_step(s, k_pool=x.k_pool, v_pool=x.v_pool, tables=x.block_tables,
                                 ctx_lens=ctx, q=x.q[t], logits=x.logits[t], h_prev=h_prev,
                                 tau=tau, temp=temp, uniforms=x.uniforms[t], params=p,
                                 block_size=16, kappa=kappa)
            done += 1
            if loop:
                h_prev[s], tau[s], temp[s], kappa[s] = o["h"], o["tau"], o["temp_next"], o["kappa"]
                ctx[s] = OAp.append_token(x.k_pool, x.v_pool, x.block_tables[s], int(ctx[s]),
                                          x.k_new[t, s], x.v_new[t, s], 16)
                t += 1
                if t < S:
                    continue
                t = 0
            s = (s + stride) % B
    return done, time.perf_counter() - t0


def cpu_baseline(x, p, seconds):
    """The float64 oracle on the host (all stages; closed loops also the
    append): one process per core of the host (sequences split between them,
    one thread each) for about `seconds`, then one thread alone for half of
    that; both scaled to whole steps per second.  Runs before the GPU is
    initialised, so the worker processes hold no device state."""
    import multiprocessing as mp
    global _BASE
    _BASE = (x, p)         # inherited by the forked workers, not pickled
    B = x.workload.batch
    n = max(1, min(len(os.sched_getaffinity(0)), 16))
    with mp.get_context("fork").Pool(n) as pool:
        res = pool.map(_oracle_worker, [(i, n, seconds) for i in range(n)])
    el = max(r[1] for r in res)
    done = sum(r[0] for r in res)
    # The one-thread figure also runs in a child: appends write the pools.
    with mp.get_context("fork").Pool(1) as pool:
        one, el1 = pool.map(_oracle_worker, [(0, 1, seconds / 2)])[0]
    if x.steps > 1:
        what = (f"{done} sequence-steps of the {x.workload.name} loop (each process runs its "
                f"sequences through consecutive loop steps from step 0, carrying the oracle's own "
                f"state and appends)")
    else:
        what = f"{done} sequence-steps of one {x.workload.name} step"
    return {"value": (done / B) / el, "unit": "steps/s", "cores": n, "kind": "oracle",
            "value_1core": (one / B) / el1,
            "sample": f"float64 oracle, all stages: {what} in {el:.1f} s over {n} processes "
                      f"(one thread each, sequences split between them), and {one} in "
                      f"{el1:.1f} s on one thread (value_1core); scaled to whole steps of "
                      f"{B} sequences"}


def counters_path(workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"decode_counters_{workload}.json")


def traffic_from_counters(workload: str):
    """HBM bytes per decode launch of this workload from committed rocprofv3
    counters, if they were taken on the current decode kernel source (else
    None)."""
    path = counters_path(workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        c = json.load(f)
    if c.get("decode_src_sha256") != decode_src_digest():
        return None
    return c.get("hbm_bytes_per_launch")


def sched_time(ent, torch, ctx, sp, b_sel, K, W):
    """Average duration of one ent_schedule call over a pool of
    ENT_SCHED_MAX_POOL sequences (seeded synthetic state)."""
    import numpy as np
    n = ent.ENT_SCHED_MAX_POOL
    rng = np.random.default_rng(1234)
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(a).to(dev)
    tau = t((rng.random(n) * 50).astype(np.float32))
    tl = t((rng.random(n) * 50).astype(np.float32))
    gain = t((rng.random(n) * 0.5).astype(np.float32))
    age = t(rng.integers(0, 40, n).astype(np.int32))
    kept = t(rng.integers(0, 512, n).astype(np.int32))
    lens = t(rng.integers(0, 32768, n).astype(np.int32))
    sel = torch.empty(n, dtype=torch.int32, device=dev)
    nsel = torch.empty(1, dtype=torch.int32, device=dev)
    pri = torch.empty(n, dtype=torch.float32, device=dev)
    prm = ent.ent_sched_params(1.0, 0.25, 4.0, 16.0, 0.5, 1e-3, 0.25)

    def call():
        ent.ent_schedule(ctx, n, prm, tau, kept, lens, tl, gain, age, b_sel, sel, nsel, pri, sp)

    for _ in range(W):
        call()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(torch.cuda.current_stream())
    for _ in range(K):
        call()
    e1.record(torch.cuda.current_stream())
    torch.cuda.synchronize()
    return {"pool": n, "b_sel": b_sel, "avg_launch_us": round(e0.elapsed_time(e1) / K * 1e3, 2)}


def calibrate_copy(torch, dev):
    """A plain 1 GiB device copy: profilers' byte counters for this kernel
    calibrate those taken on the step's kernels."""
    src = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def closed_loop(args, w, p):
    """A closed-loop workload: every loop step is one ent_decode_step_append
    call (the decode step, then the append of the new token's K/V), the
    controller state and the kept-fraction state carried on the device, fresh
    logits, queries and uniforms per step.  --warmup loop steps run untimed, then --steps
    consecutive loop steps are timed between two events (a pass past the
    workload's last step starts the loop over from its initial state: lengths,
    controller state, kept-fraction state and the appended blocks' summaries
    restored by device copies).

    A second, untimed pass replays the same steps from the initial state
    (the loop is deterministic) and records each timed step's kept lists and
    lengths, for the byte count and for the roofline pass: the decode entry
    point (attention plus segment merge) issued once per timed step, back to
    back between two events, on that step's queries, kept lists and lengths
    (the pools then hold later appended tokens too, past those lengths,
    which the decode never reads)."""
    import torch

    from paper_2603_03310_amd import ent
    from synth import generate
    from synth.device import config_fields, upload

    t0 = time.perf_counter()
    x = generate(w)
    print(f"[bench] generated {w.name} ({w.steps} steps) in {time.perf_counter() - t0:.1f} s",
          file=sys.stderr, flush=True)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(x, p, args.cpu_seconds)
        print("[bench] cpu baseline done", file=sys.stderr, flush=True)
    ent.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    d = upload(x, dev)
    B, S = w.batch, w.steps
    K, W = args.steps, args.warmup
    cfg = ent.ent_config()
    for k, v in config_fields(w, p, x.num_pool_blocks).items():
        setattr(cfg, k, v)
    ctx = ent.ent_init(cfg)
    sp = torch.cuda.current_stream().cuda_stream
    ent.ent_block_summary(ctx, B, d.k_pool, d.block_tables, d.ctx_lens, d.ksum, sp)
    ld = x.logits.shape[2]
    init = [torch.from_numpy(a).to(dev) for a in (x.h_prev, x.tau, x.temp, x.ctx_lens)]
    # Summaries of every block a pass of appends touches (the blocks holding
    # positions ctx_len .. ctx_len + S - 1), saved to restore them.
    touched = sorted({int(x.block_tables[s][j])
                      for s in range(B)
                      for j in range(int(x.ctx_lens[s]) // 16, (int(x.ctx_lens[s]) + S - 1) // 16 + 1)})
    touched = torch.tensor(touched, dtype=torch.long, device=dev)
    ksum_saved = d.ksum.index_select(0, touched)

    def reset():
        for dst, src in zip((d.h_prev, d.tau, d.temp, d.ctx_lens), init):
            dst.copy_(src)
        d.kappa.fill_(float("nan"))
        d.ksum.index_copy_(0, touched, ksum_saved)

    def step(t):
        if t % S == 0 and t > 0:
            reset()
        i = t % S
        ent.ent_decode_step_append(ctx, B, d.logits[i], ld, d.h_prev, d.tau, d.temp, d.q[i],
                                   d.k_pool, d.v_pool, d.ksum, d.block_tables, d.ctx_lens,
                                   d.uniforms[i], d.k_new[i], d.v_new[i], d.h, d.temp_used, d.kept,
                                   d.n_kept, d.out, d.tokens, d.row_stats, d.lse, None, None, sp,
                                   d.kappa)

    if args.calibrate_copy:
        calibrate_copy(torch, dev)
    # Pass A: W warm-up loop steps, then K timed consecutive loop steps.
    for t in range(W):
        step(t)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record()
    for t in range(W, W + K):
        step(t)
    e1.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_wall) * 1e3
    ms_step = e0.elapsed_time(e1) / K
    flags = ent.ent_device_status(ctx, sp)
    if flags:
        raise SystemExit(f"device flags raised: {flags}")
    print(f"[bench] timed {K} loop steps after {W} warm-up steps", file=sys.stderr, flush=True)

    # Pass B (untimed): the same steps from the initial state; each timed
    # step's kept lists, counts and lengths are kept on the device.
    reset()
    elem = w.elem_bytes
    kv_kept, blocks_kept, blocks_all, all_bytes = 0, 0, 0, 0
    rec_kept = torch.empty((K,) + tuple(d.kept.shape), dtype=torch.int32, device=dev)
    rec_nk = torch.empty((K, B), dtype=torch.int32, device=dev)
    rec_ctx = torch.empty((K, B), dtype=torch.int32, device=dev)
    dec_bytes = 0
    Hq, hd = w.num_q_heads, w.head_dim
    xs = type("X", (), {})()
    xs.workload = w
    for t in range(W + K):
        if t >= W:
            if t % S == 0 and t > 0:
                reset()
            rec_ctx[t - W].copy_(d.ctx_lens)
            xs.ctx_lens = d.ctx_lens.cpu().numpy()
        step(t)
        if t < W:
            continue
        torch.cuda.synchronize()
        rec_kept[t - W].copy_(d.kept)
        rec_nk[t - W].copy_(d.n_kept)
        nk, kp = d.n_kept.cpu().numpy(), d.kept.cpu().numpy()
        kv_step = kv_bytes_kept(xs, nk, kp, elem)
        kv_kept += kv_step
        all_bytes += total_bytes(w, xs.ctx_lens, kv_step, elem, p.scoring)
        blocks_kept += int(nk.sum())
        blocks_all += int(sum(-(-int(n) // 16) for n in xs.ctx_lens))
        dec_bytes += (kv_step + B * Hq * hd * elem + B * Hq * hd * 4 + B * Hq * 4
                      + 2 * 4 * int(nk.sum()) + 4 * B)

    # Pass C: the roofline kernel's entry point, once per timed step (its
    # queries, kept lists and lengths), back to back between two events on
    # the launch stream; W warm-up calls first.
    def decode_call(j):
        i = (W + j) % S
        ent.ent_sparse_paged_decode(ctx, B, d.q[i], d.k_pool, d.v_pool, d.block_tables,
                                    rec_ctx[j], rec_kept[j], rec_nk[j], d.out, d.lse, sp)

    for j in range(min(W, K)):
        decode_call(j)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for j in range(K):
        decode_call(j)
    c1.record()
    torch.cuda.synchronize()
    dec_us = c0.elapsed_time(c1) / K * 1e3
    flags = ent.ent_device_status(ctx, sp)
    if flags:
        raise SystemExit(f"device flags raised: {flags}")
    ent.ent_destroy(ctx)

    metric_bytes = kv_kept / K + 4 * B * w.vocab
    gbps = metric_bytes / (ms_step * 1e-3) / 1e9
    dec_per_launch = dec_bytes / K
    achieved = dec_per_launch / (dec_us * 1e-6) / 1e9
    line = {
        "metric": METRIC, "value": round(1e3 / ms_step, 3), "unit": "steps/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(ms_step, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.kv_dtype,
        "data": "synthetic (seeded; shapes and value recipes of the workload)",
        "config": {"workload": w.name, "batch": B, "q_heads": Hq, "kv_heads": w.num_kv_heads,
                   "head_dim": hd, "block_size": 16, "ctx": list(w.ctx), "vocab": w.vocab,
                   "kv_dtype": w.kv_dtype, "loop_steps": S, "timed_loop_steps": [W, W + K],
                   "step": "ent_decode_step_append", "entropy": args.estimator},
        "hbm_gbps_kept_kv_plus_logits": round(gbps, 1),
        "hbm_frac_kept_kv_plus_logits": round(gbps / HBM_PEAK_GBPS, 4),
        "metric_bytes_per_step": int(metric_bytes),
        "total_bytes_per_step": int(all_bytes / K),
        "hbm_gbps_total": round(all_bytes / K / (ms_step * 1e-3) / 1e9, 1),
        "hbm_frac_total": round(all_bytes / K / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        "kept_block_fraction": round(blocks_kept / max(1, blocks_all), 4),
        "wall_ms_per_step": round(wall_ms / K, 5),
        "roofline": {"kernel": "sparse_paged_decode", "bound": "hbm",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic_from_counters(w.name),
                     "bytes_per_launch": int(dec_per_launch), "avg_launch_us": round(dec_us, 2)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2603_03310_amd import ent
    from synth import WORKLOADS, default_params, generate
    from synth.device import config_fields, upload

    if not os.path.exists(ent.LIB_PATH):
        ent.load()        # raises: the library has not been built (no fallback)
    w = WORKLOADS[args.workload]
    if args.q_heads:
        w = w.replace(num_q_heads=args.q_heads, name=f"{w.name}_q{args.q_heads}")
    p = default_params(w)
    est = {"exact": 0, "topk": 1, "tail": 2}[args.estimator]
    if est:
        p = p.replace(estimator=est, est_k=args.est_k)
    if args.eps_h is not None:
        p = p.replace(eps_h=args.eps_h)
    p = p.replace(scoring=1 if args.scoring == "exact" else 0, keep_first=args.keep_first,
                  keep_last=args.keep_last)
    if w.steps != 1:
        return closed_loop(args, w, p)
    t0 = time.perf_counter()
    x = generate(w)
    print(f"[bench] generated {w.name} in {time.perf_counter() - t0:.1f} s", file=sys.stderr,
          flush=True)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(x, p, args.cpu_seconds)
        print("[bench] cpu baseline done", file=sys.stderr, flush=True)
    ent.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    copies = [upload(x, dev) for _ in range(max(1, args.copies))]
    B = w.batch
    K, W = args.steps, args.warmup
    nslots = K + W
    init = torch.stack([torch.from_numpy(x.h_prev), torch.from_numpy(x.tau),
                        torch.from_numpy(x.temp)]).to(dev)
    states = [init.unsqueeze(0).repeat(nslots, 1, 1).contiguous() for _ in range(2)]
    cfg = ent.ent_config()
    for k, v in config_fields(w, p, x.num_pool_blocks).items():
        setattr(cfg, k, v)
    ctx = ent.ent_init(cfg)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    for c in copies:
        ent.ent_block_summary(ctx, B, c.k_pool, c.block_tables, c.ctx_lens, c.ksum, sp)
    o = copies[0]          # outputs shared by all copies
    ld = x.logits.shape[2]

    def issue_fused(i, st):
        c = copies[i % len(copies)]
        ent.ent_decode_step(ctx, B, c.logits[0], ld, st[i, 0], st[i, 1], st[i, 2], c.q[0],
                            c.k_pool, c.v_pool, c.ksum, c.block_tables, c.ctx_lens,
                            c.uniforms[0], o.h, o.temp_used, o.kept, o.n_kept, o.out, o.tokens,
                            o.row_stats, o.lse, None, None, sp)

    def issue_staged(i, st, ev):
        c = copies[i % len(copies)]
        hp, ta, te = st[i, 0], st[i, 1], st[i, 2]
        ev[0].record(stream)
        ent.ent_entropy_temperature(ctx, B, c.logits[0], ld, hp, ta, te, o.h, o.temp_used,
                                    o.row_stats, sp)
        ev[1].record(stream)
        ent.ent_block_select(ctx, B, c.q[0], c.ksum, c.block_tables, c.ctx_lens, o.h, o.kept,
                             o.n_kept, None, None, sp, None, c.k_pool)
        ev[2].record(stream)
        ent.ent_sparse_paged_decode(ctx, B, c.q[0], c.k_pool, c.v_pool, c.block_tables,
                                    c.ctx_lens, o.kept, o.n_kept, o.out, o.lse, sp)
        ev[3].record(stream)
        ent.ent_sample(ctx, B, c.logits[0], ld, o.row_stats, o.temp_used, c.uniforms[0],
                       o.tokens, sp)
        ev[4].record(stream)

    if args.calibrate_copy:
        calibrate_copy(torch, dev)

    # Pass A: the timed steps (ent_decode_step), nothing between the launches.
    for i in range(W):
        issue_fused(i, states[0])
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record(stream)
    for i in range(W, W + K):
        issue_fused(i, states[0])
    e1.record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_wall) * 1e3
    ms_step = e0.elapsed_time(e1) / K

    # Pass B: the same steps through the four per-stage entry points, with an
    # event around each (per-stage times; the decode entry point is the
    # roofline kernel's launch: attention plus the merge of split segments).
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(K + W)]
    for i in range(W):
        issue_staged(i, states[1], evs[K + i])
    for i in range(K):
        issue_staged(W + i, states[1], evs[i])
    torch.cuda.synchronize()
    names = ["entropy_temperature", "block_select", "sparse_paged_decode", "sample"]
    per_k = {n: float(np.mean([evs[i][j].elapsed_time(evs[i][j + 1]) for i in range(K)])) * 1e3
             for j, n in enumerate(names)}
    # Pass C: the roofline kernel's entry point (decode attention plus the
    # merge of split segments) issued K times back to back on the same stream,
    # bracketed by two events, on the kept lists of the last staged step
    # (every copy holds the same data): its average launch duration without
    # the gap an event between calls adds.
    for i in range(W):
        c = copies[i % len(copies)]
        ent.ent_sparse_paged_decode(ctx, B, c.q[0], c.k_pool, c.v_pool, c.block_tables,
                                    c.ctx_lens, o.kept, o.n_kept, o.out, o.lse, sp)
    d0, d1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    d0.record(stream)
    for i in range(K):
        c = copies[(W + i) % len(copies)]
        ent.ent_sparse_paged_decode(ctx, B, c.q[0], c.k_pool, c.v_pool, c.block_tables,
                                    c.ctx_lens, o.kept, o.n_kept, o.out, o.lse, sp)
    d1.record(stream)
    torch.cuda.synchronize()
    dec_us = d0.elapsed_time(d1) / K * 1e3
    # Pass D: the scheduler that picks the next batch (Section 3.1), over the
    # largest pool of active sequences, selecting this workload's batch; K
    # calls back to back between two events.
    sched = sched_time(ent, torch, ctx, sp, B, K, W)
    flags = ent.ent_device_status(ctx, sp)
    if flags:
        raise SystemExit(f"device flags raised: {flags}")

    n_kept = o.n_kept.cpu().numpy()
    kept = o.kept.cpu().numpy()
    elem = 2 if w.kv_dtype == "bf16" else 4
    kv_kept = kv_bytes_kept(x, n_kept, kept, elem)
    logit_bytes = 4 * B * w.vocab
    metric_bytes = kv_kept + logit_bytes
    all_bytes = total_bytes(w, x.ctx_lens, kv_kept, elem, p.scoring)
    nb_tot = int(sum(-(-int(n) // 16) for n in x.ctx_lens))
    kept_frac = float(n_kept.sum()) / max(1, nb_tot)
    steps_per_s = 1e3 / ms_step
    gbps = metric_bytes / (ms_step * 1e-3) / 1e9

    # Decode kernel roofline: algorithmic bytes of one launch / its average duration.
    Hq, d = w.num_q_heads, w.head_dim
    dec_bytes = (kv_kept + B * Hq * d * elem + B * Hq * d * 4 + B * Hq * 4
                 + 2 * 4 * int(n_kept.sum()) + 4 * B)
    achieved = dec_bytes / (dec_us * 1e-6) / 1e9
    ent.ent_destroy(ctx)

    line = {
        "metric": METRIC, "value": round(steps_per_s, 3), "unit": "steps/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(ms_step, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.kv_dtype,
        "data": "synthetic (seeded; shapes and value recipes of the workload)",
        "config": {"workload": w.name, "batch": B, "q_heads": Hq, "kv_heads": w.num_kv_heads,
                   "head_dim": d, "block_size": 16, "ctx": list(w.ctx), "vocab": w.vocab,
                   "kv_dtype": w.kv_dtype, "entropy": args.estimator,
                   **({"est_k": args.est_k} if est else {}),
                   **({"eps_h": p.eps_h} if p.eps_h else {}),
                   **({"scoring": args.scoring} if p.scoring else {}),
                   **({"keep_first": p.keep_first} if p.keep_first else {}),
                   **({"keep_last": p.keep_last} if p.keep_last else {})},
        "hbm_gbps_kept_kv_plus_logits": round(gbps, 1),
        "hbm_frac_kept_kv_plus_logits": round(gbps / HBM_PEAK_GBPS, 4),
        "metric_bytes_per_step": int(metric_bytes),
        "total_bytes_per_step": int(all_bytes),
        "hbm_gbps_total": round(all_bytes / (ms_step * 1e-3) / 1e9, 1),
        "hbm_frac_total": round(all_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        "kept_block_fraction": round(kept_frac, 4),
        "per_stage_us": {k: round(v, 2) for k, v in per_k.items()},
        "staged_ms_per_step": round(sum(per_k.values()) * 1e-3, 5),
        "wall_ms_per_step": round(wall_ms / K, 5),
        "roofline": {"kernel": "sparse_paged_decode", "bound": "hbm",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic_from_counters(w.name),
                     "bytes_per_launch": int(dec_bytes), "avg_launch_us": round(dec_us, 2)},
        "cpu_baseline": cpu,
        "schedule": sched,
    }
    if p.scoring:
        # The exact mode reads every valid key once inside the block selection.
        k_all = int(sum(int(n) for n in x.ctx_lens)) * w.num_kv_heads * w.head_dim * elem
        sel_us = per_k["block_select"]
        line["exact_scoring"] = {"k_bytes": k_all, "block_select_us": round(sel_us, 2),
                                 "gbps_on_k": round(k_all / (sel_us * 1e-6) / 1e9, 1)}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
