#!/usr/bin/env python3
"""Throughput of the StepKV compression pass on one MI355X.

One step = the whole pass over one synthetic batch at one pruning boundary:
host step-utility update for the newest step of every sequence (Algorithm 1
phases 1-2, from the state of the boundaries before it; it runs on the host
while the GPU computes the saliency, which does not depend on it) ->
saliency -> priority -> top-B select -> K/V compaction, all layers and KV
heads. Inputs are resident in HBM before the timed region. Prints one JSON
line.

Before the warmup, untimed: a pass of K steps writes --flush-mib bytes before
each step (evicting the Infinity Cache) and times every step from the cold cache
with its own events ("flushed"); "hbm_ceilings" gives the read and copy
bandwidth of plain streaming kernels with the compaction's access width;
"mfma_issue" gives the bf16 MFMA rate of a probe at the sweeps' occupancy, alone
and with the sweeps' vector work per MFMA (an exp2, an FMA and an add for each
of two score elements), and their ratio, the share of MFMA issue that mix
leaves. This work also lets the board's power management settle before the
timed steps.
Then W warmup steps and the K timed steps, which carry no event inside a step.
Per-stage times (HIP events around each C ABI call, on the launch stream) and
the saliency roofline come from a second pass of the same K steps.

By default the saliency is computed from the window queries and the cache
alone (two sweeps over K). With --lse-fed the window rows' log-sum-exps are
an input, as the observation prefill's attention provides them (App. C.2),
and the saliency takes one sweep.

    python bench.py [--steps K] [--warmup W] [--workload l32_32k] [--budget 1024] [--lse-fed]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "KV tokens compressed/sec (all layers) + achieved HBM GB/s vs peak, 32k ctx"
HBM_PEAK_GBS = 8000.0      # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="l32_32k")
    ap.add_argument("--budget", type=int, default=None)
    ap.add_argument("--window", type=int, default=None)
    ap.add_argument("--layers", type=int, default=None)
    ap.add_argument("--seed", type=int, default=233)
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="budget for the oracle CPU baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--lse-fed", action="store_true",
                    help="take the window rows' log-sum-exps as an input (one sweep over K)")
    ap.add_argument("--schedule", type=int, choices=(0, 1, 2), default=0,
                    help="saliency sweeps: 0 chosen per problem, 1 one launch per sweep, "
                         "2 both in one launch (stepkv_params.saliency_schedule)")
    ap.add_argument("--causal-tail", action="store_true",
                    help="window slot w sees keys up to N - W + w only (causal prefill)")
    ap.add_argument("--text-signals", action="store_true",
                    help="derive each boundary's step signals from synthetic trajectory text "
                         "(host engine) instead of drawing them")
    ap.add_argument("--decode", action="store_true",
                    help="add one decode step over the compacted cache (every layer and query "
                         "head, random queries) to each step, as its own stage")
    ap.add_argument("--selector", choices=("stepkv", "token-only", "last-query"), default="stepkv",
                    help="token-only: the pooled window saliency alone (beta = 0, SnapKV-style); "
                         "last-query: one window query, no pooling, beta = 0 (TOVA-style)")
    ap.add_argument("--shared-layers", type=int, default=0,
                    help="shared-index mode: rank each sequence once from the saliency of its "
                         "last N layers and compact every layer and head with that one set")
    ap.add_argument("--flush-mib", type=int, default=1024,
                    help="bytes written before each step of the flushed timing pass (evicts the "
                         "256 MB Infinity Cache); 0 skips that pass")
    ap.add_argument("--ceiling-mib", type=int, default=1024,
                    help="buffer size of the HBM read and copy ceiling probes; 0 skips them")
    ap.add_argument("--issue-probe-iters", type=int, default=4000,
                    help="loops of the MFMA issue-rate probe (MFMAs alone, then with the "
                         "saliency sweeps' vector work per MFMA); 0 skips it")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="run one plain device copy of this size (HBM counter calibration)")
    ap.add_argument("--record-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc counter_collection.csv files (FETCH_SIZE, "
                         "WRITE_SIZE) of a --copy-probe-mib run into profiles/traffic.json")
    return ap.parse_args()


# saliency-stage kernels: both sweeps in one launch (after its counters are cleared), or the
# per-sweep kernels with the LSE combine or import (the one-launch name comes first: it does
# not contain the per-sweep kernel's name)
SALIENCY_KERNELS = ("saliency_fused_kernel", "saliency_kernel", "lse_combine_kernel",
                    "lse_import_kernel", "fill_u32_kernel")


def _saliency_part(name: str, lse_fed: bool):
    """The saliency-stage kernel a dispatch belongs to, or None. With lse_fed the
    row-LSE sweep and its combine belong to the untimed prefill stand-in."""
    import re

    for k in SALIENCY_KERNELS:
        if k in name:
            first_sweep = k == "saliency_kernel" and re.search(r"saliency_kernel<\d+, \d+, 1[,>]", name)
            if lse_fed and (k == "lse_combine_kernel" or first_sweep):
                return None
            return k
    return None


def record_traffic(args) -> None:
    """HBM bytes per saliency launch, scaled by the counters' reading of a plain copy."""
    import csv
    import re
    from collections import defaultdict

    def per_dispatch(path, counter):
        vals = defaultdict(float)
        names = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            vals[r["Dispatch_Id"]] += float(r["Counter_Value"])  # KiB, summed over instances
            names[r["Dispatch_Id"]] = r["Kernel_Name"]
        return vals, names

    probe = args.copy_probe_mib << 20
    if probe <= 0:
        sys.exit("--record-traffic needs the --copy-probe-mib size the counters were taken with")
    out = {}
    for counter, path in (("FETCH_SIZE", args.record_traffic[0]),
                          ("WRITE_SIZE", args.record_traffic[1])):
        vals, names = per_dispatch(path, counter)
        copies = [d for d in vals if "copyBuffer" in names[d]]
        cal = probe / (max(vals[d] for d in copies) * 1024.0)  # bytes per counted byte
        per_kernel = defaultdict(list)
        launches = 0  # saliency stages: each runs the column-sum sweep exactly once
        for d, v in vals.items():
            k = _saliency_part(names[d], args.lse_fed)
            if k is None:
                continue
            per_kernel[k].append(v * 1024.0 * cal)
            launches += bool(re.search(r"saliency_kernel<\d+, \d+, 2[,>]|saliency_fused_kernel<",
                                       names[d]))
        out[counter] = {"calibration": cal, "launches": launches,
                        "bytes": sum(sum(v) for v in per_kernel.values()) / launches,
                        "per_kernel": {k: sum(v) / launches for k, v in per_kernel.items()}}
    budget = args.budget or 1024
    key = traffic_key(args.workload, budget, args.window or 64, args.lse_fed, args.shared_layers,
                      args.schedule)
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        db = json.load(open(path))
    except (OSError, ValueError):
        db = {}
    db[key] = {
        "saliency_source_sha256": source_digest(),
        "hbm_bytes_per_launch": round(out["FETCH_SIZE"]["bytes"] + out["WRITE_SIZE"]["bytes"]),
        "fetch_bytes_per_launch": round(out["FETCH_SIZE"]["bytes"]),
        "write_bytes_per_launch": round(out["WRITE_SIZE"]["bytes"]),
        "fetch_calibration": out["FETCH_SIZE"]["calibration"],
        "write_calibration": out["WRITE_SIZE"]["calibration"],
        "per_kernel_fetch_bytes": out["FETCH_SIZE"]["per_kernel"],
        "per_kernel_write_bytes": out["WRITE_SIZE"]["per_kernel"],
        "copy_probe_bytes": probe,
    }
    with open(path, "w") as f:
        json.dump(db, f, indent=1, sort_keys=True)
    print(json.dumps(db[key]))


def source_digest() -> str:
    """sha256 of the saliency kernel source: traffic figures are valid for it only."""
    import hashlib

    path = os.path.join(ROOT, "paper_2609_22158_amd", "csrc", "saliency.hip")
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def traffic_key(workload: str, budget: int, window: int, lse_fed: bool, shared_layers: int = 0,
                schedule: int = 0) -> str:
    """Key of a traffic record: the workload and every option that changes the
    saliency launches (shared-index mode sweeps only its last layers; a forced
    schedule may read K from HBM twice)."""
    return (f"{workload}_b{budget}_w{window}" + ("_lse" if lse_fed else "")
            + (f"_shared{shared_layers}" if shared_layers > 0 else "")
            + (f"_schedule{schedule}" if schedule else ""))


def recorded_traffic(key: str):
    """HBM bytes per saliency launch from the committed counter runs, or None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f).get(key)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("saliency_source_sha256") != source_digest():
        return None  # kernel changed since the counters were taken
    return rec.get("hbm_bytes_per_launch")


def cpu_baseline(w, budget, seconds, params, lse_fed=False):
    """Time the oracle on whole (sequence, layer, KV head) triples until `seconds` pass.

    With lse_fed the oracle takes each triple's row log-sum-exps as given (computed
    beforehand by the oracle itself, outside the timed region)."""
    import oracle as O

    try:
        from threadpoolctl import threadpool_info

        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    S = np.concatenate([O.run_step_updates(g.valid, g.gain, g.red, g.obs_sim.astype(np.float64),
                                           O.Params())[2] for g in w.signals])
    triples = [(s, l, h) for l in range(w.num_layers) for h in range(w.num_kv_heads)
               for s in range(w.num_seqs)]
    rng = np.random.default_rng(0)
    rng.shuffle(triples)
    op = O.Params(alpha=params.alpha, beta=params.beta, pool_kernel=params.pool_kernel,
                  causal_tail=bool(params.causal_tail))
    G = w.num_q_heads // w.num_kv_heads
    lse_win = np.zeros(w.q_win.shape[:4]) if lse_fed else None
    done, tokens, dt = 0, 0, 0.0
    for s, l, h in triples:
        if lse_fed:  # the prefill's output, not part of the timed work
            a, b = int(w.cu_seqlens[s]), int(w.cu_seqlens[s + 1])
            rows = O.window_rows(O.decode_bf16(w.q_win[l, s]), h, G)
            vis = O.visible_keys(b - a, w.window, G, op.causal_tail)
            lse = O.window_row_lse(rows, O.decode_bf16(w.k[l, h, a:b]),
                                   1.0 / math.sqrt(w.head_dim), vis)
            lse_win[l, s, :, h * G:(h + 1) * G] = lse.reshape(w.window, G)
        t0 = time.perf_counter()
        O.compress(w.q_win, w.k, w.v, w.cu_seqlens, w.step_ids, w.protected, w.cu_steps, S,
                   budget, op, layers=[l], heads=[h], seqs=[s], lse_win=lse_win)
        dt += time.perf_counter() - t0
        done += 1
        tokens += w.seqlens[s]
        if dt >= seconds:
            break
    # whole-job rate: every token is scored in all L x Hkv heads
    per_head_rate = tokens / dt
    value = per_head_rate / (w.num_layers * w.num_kv_heads)
    return {"value": value, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "host_cpus": os.cpu_count(),
            "sample": f"{done} of {len(triples)} (sequence, layer, KV head) triples "
                      f"({tokens} token-heads) in {dt:.1f} s, scaled to all {w.num_layers} layers "
                      f"x {w.num_kv_heads} KV heads"}


def cpu_baseline_shared(w, budget, seconds, params, last_layers):
    """Time the oracle's shared-index pass, one sequence at a time, until `seconds` pass."""
    import oracle as O

    try:
        from threadpoolctl import threadpool_info

        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    S = np.concatenate([O.run_step_updates(g.valid, g.gain, g.red, g.obs_sim.astype(np.float64),
                                           O.Params())[2] for g in w.signals])
    op = O.Params(alpha=params.alpha, beta=params.beta, pool_kernel=params.pool_kernel,
                  causal_tail=bool(params.causal_tail))
    done, tokens, dt = 0, 0, 0.0
    for s in range(w.num_seqs):
        t0 = time.perf_counter()
        O.compress_shared(w.q_win, w.k, w.v, w.cu_seqlens, w.step_ids, w.protected, w.cu_steps,
                          S, budget, op, last_layers=last_layers, seqs=[s])
        dt += time.perf_counter() - t0
        done += 1
        tokens += w.seqlens[s]
        if dt >= seconds:
            break
    return {"value": tokens / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "host_cpus": os.cpu_count(),
            "sample": f"{done} of {w.num_seqs} sequence(s) ({tokens} tokens), shared-index pass "
                      f"over the last {last_layers} layers and all {w.num_layers} layers' "
                      f"compaction, in {dt:.1f} s"}


def main():
    args = parse()
    if args.record_traffic:
        record_traffic(args)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus} GPUs, WORLD_SIZE={world}): "
              "the compression pass is independent per (layer, KV head) and this build has no "
              "multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    from synth import make_workload

    t_gen = time.perf_counter()
    kw = {}
    if args.window:
        kw["window"] = args.window
    if args.selector == "last-query":
        kw["window"] = 1
    if args.layers:
        kw["num_layers"] = args.layers
    w = make_workload(args.workload, args.seed, **kw)
    budget = args.budget or w.budget
    print(f"# generated {args.workload} in {time.perf_counter() - t_gen:.1f} s", file=sys.stderr,
          flush=True)

    import torch

    from paper_2609_22158_amd import binding as B

    dev = "cuda:0"
    torch.cuda.set_device(0)
    # no device status word: its checks are a diagnostic, not part of the timed pass
    pb = B.Problem.from_workload(w, dev, status=False)
    q, k, v = (B.bf16_from_bits(x, dev) for x in (w.q_win, w.k, w.v))
    sid = torch.from_numpy(w.step_ids).to(dev)
    prot = torch.from_numpy(w.protected).to(dev)
    util = torch.empty(pb.total_steps, dtype=torch.float32, device=dev)
    # one pinned staging row per step of the run (flushed pass, warmup, timed pass,
    # stage-timing pass), so that the host never overwrites a row whose copy may
    # still be queued and no event has to be waited on inside a step
    n_rows = args.warmup + 3 * args.steps
    util_pinned = torch.empty((n_rows, max(pb.total_steps, 1)), dtype=torch.float32,
                              pin_memory=True)
    slot = [0]
    L, Hkv, ntot, d = w.num_layers, w.num_kv_heads, w.total_tokens, w.head_dim
    sal = torch.empty((L, Hkv, ntot), dtype=torch.float32, device=dev)
    scores = torch.empty_like(sal)
    idx = torch.empty((L, Hkv, ntot), dtype=torch.int32, device=dev)
    cu_ret = torch.empty(w.num_seqs + 1, dtype=torch.int32, device=dev)
    out_rows = int(pb.retained_rows(w.protected, budget)[-1])
    k_out = torch.empty((L, Hkv, out_rows, d), dtype=torch.bfloat16, device=dev)
    v_out = torch.empty_like(k_out)
    ws = torch.empty(pb.saliency_workspace_bytes(), dtype=torch.uint8, device=dev)
    sched = dict(saliency_schedule=args.schedule)
    if args.selector == "token-only":
        params = B.Params.token_only(causal_tail=int(args.causal_tail), **sched)
    elif args.selector == "last-query":
        params = B.Params.last_query_only(causal_tail=int(args.causal_tail), **sched)
    else:
        params = B.Params(causal_tail=int(args.causal_tail), **sched)
    stream = torch.cuda.current_stream()
    lse = None
    if args.lse_fed:  # stands for the prefill attention's row LSE, resident in HBM
        lse = B.window_lse(pb, q, k, params, workspace=ws)
        torch.cuda.synchronize()

    # a0 state: every trajectory's step utilities up to the boundary before its last step
    trackers, snaps, texts = [], [], []
    for i, g in enumerate(w.signals):
        if args.text_signals:  # the signals come from each step's text
            from synth.text import make_text_trajectory

            steps = make_text_trajectory(args.seed + 7919 * i, g.num_steps)
            tr = B.TextTracker(g.num_steps)
            for t in range(g.num_steps - 1):
                tr.update(*steps[t])
            texts.append(steps[-1])
        else:
            tr = B.StepTracker(g.num_steps)
            for t in range(g.num_steps - 1):
                tr.update(g.valid[t], g.gain[t], g.red[t], g.obs_sim[t, :t])
        trackers.append(tr)
        snaps.append(tr.snapshot())
    util_host = util_pinned.numpy()
    cu_steps = [int(x) for x in w.cu_steps]

    def host_update():
        # a0: the boundary after each sequence's newest step (Algorithm 1 phases 1-2)
        b = slot[0]
        slot[0] += 1
        for i, (g, tr) in enumerate(zip(w.signals, trackers)):
            tr.restore(snaps[i])  # every timed step redoes the same boundary
            out = util_host[b, cu_steps[i]:cu_steps[i + 1]]
            if args.text_signals:
                tr.update(*texts[i], out=out)
            else:
                t = g.num_steps - 1
                tr.update(g.valid[t], g.gain[t], g.red[t], g.obs_sim[t, :t], out=out)
        util.copy_(util_pinned[b, :pb.total_steps], non_blocking=True)

    if args.decode:  # one decode query per (layer, sequence, query head)
        qd_bits = np.random.default_rng(args.seed + 1).standard_normal(
            (L, w.num_seqs, w.num_q_heads, d)).astype(np.float32)
        from synth import f32_to_bf16_bits

        q_dec = B.bf16_from_bits(f32_to_bf16_bits(qd_bits), dev)
        dec_out = torch.empty((L, w.num_seqs, w.num_q_heads, d), dtype=torch.float32, device=dev)
        dec_ws = torch.empty(max(int(B.load().stepkv_decode_workspace_bytes(
            B.ctypes.byref(pb.c), out_rows)), 1), dtype=torch.uint8, device=dev)

    def decode(ev, i):
        if args.decode:
            B.decode_attention(pb, q_dec, k_out, v_out, cu_ret, out_rows, workspace=dec_ws,
                               out=dec_out)
            if ev:
                ev[i].record(stream)

    def step(ev=None):
        if ev:
            ev[0].record(stream)
        if lse is None:
            B.saliency(pb, q, k, params, workspace=ws, out=sal)
        else:
            B.saliency_from_lse(pb, q, k, lse, params, workspace=ws, out=sal)
        host_update()  # on the host while the GPU runs the saliency, which does not need S
        if ev:
            ev[1].record(stream)
        B.priority(pb, sal, sid, prot, util, params, scores=scores)
        if ev:
            ev[2].record(stream)
        B.select(pb, scores, prot, sid, budget, idx=idx, cu_retained=cu_ret)
        if ev:
            ev[3].record(stream)
        B.compact(pb, k, v, idx, cu_ret, out_rows, k_out=k_out, v_out=v_out)
        if ev:
            ev[4].record(stream)
        decode(ev, 5)

    shared = args.shared_layers > 0
    if shared:
        n_sh = min(args.shared_layers, L)
        scores_sh = torch.empty(ntot, dtype=torch.float32, device=dev)
        idx_sh = torch.empty(ntot, dtype=torch.int32, device=dev)
        ws_sh = torch.empty(max(int(B.load().stepkv_score_shared_workspace_bytes(
            B.ctypes.byref(pb.c), n_sh)), 1), dtype=torch.uint8, device=dev)

        def step(ev=None):  # noqa: F811 - the shared-index pass
            host_update()
            if ev:
                ev[0].record(stream)
            B.score_shared(pb, q, k, sid, prot, util, params, last_layers=n_sh, lse=lse,
                           workspace=ws_sh, scores=scores_sh)
            if ev:
                ev[1].record(stream)
            B.select_shared(pb, scores_sh, prot, sid, budget, idx=idx_sh, cu_retained=cu_ret)
            if ev:
                ev[2].record(stream)
            B.compact_shared(pb, k, v, idx_sh, cu_ret, out_rows, k_out=k_out, v_out=v_out)
            if ev:
                ev[3].record(stream)
            decode(ev, 4)

    # Untimed measurements first: the cold-cache pass and the ceiling and issue
    # probes run before the warmup, so that the board's power management has
    # settled when the timed steps start. After idle the first launches run at
    # boost clocks, then the board throttles to its power limit, undershoots and
    # recovers over some 25 ms of load (the sweeps' launches 3-5 of a bench run
    # take 1.40-1.49 ms, the later ones 1.06-1.15 ms); a pass that runs
    # continuously sees the settled clocks.
    # flushed pass: a write of --flush-mib before every step evicts the Infinity
    # Cache, and per-step events time each step from a cold cache
    flushed = None
    if args.flush_mib > 0:
        flush_buf = torch.empty(args.flush_mib << 20, dtype=torch.uint8, device=dev)
        fl_ms = []
        for i in range(args.steps):
            flush_buf.fill_(i & 0xFF)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            step()
            e1.record(stream)
            e1.synchronize()
            fl_ms.append(e0.elapsed_time(e1))
        del flush_buf
        q10, q50, q90 = np.percentile(fl_ms, [10, 50, 90])
        flushed = {"ms_per_step_median": round(float(q50), 4), "p10": round(float(q10), 4),
                   "p90": round(float(q90), 4), "flush_bytes": args.flush_mib << 20,
                   "value_median": round(float(ntot) / (q50 * 1e-3), 1)}
    ceilings = None
    if args.ceiling_mib > 0:  # plain streaming kernels with the compaction's access width
        nb = args.ceiling_mib << 20
        src_buf = torch.ones(nb, dtype=torch.uint8, device=dev)
        dst_buf = torch.empty(nb, dtype=torch.uint8, device=dev)
        res = {}
        for name, copy in (("read", False), ("copy", True)):
            for _ in range(3):
                B.bandwidth_probe(src_buf, dst_buf, copy)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            reps = 20
            e0.record(stream)
            for _ in range(reps):
                B.bandwidth_probe(src_buf, dst_buf, copy)
            e1.record(stream)
            e1.synchronize()
            t = e0.elapsed_time(e1) * 1e-3 / reps
            res[f"{name}_gbps"] = round(nb * (2 if copy else 1) / t / 1e9, 1)
        res["bytes"] = nb
        ceilings = res
        del src_buf, dst_buf
    issue = None
    if args.issue_probe_iters > 0:  # the MFMA rate the sweeps' instruction mix leaves
        blocks = 512  # 2 workgroups of 4 waves per CU: the sweeps' 2 waves per SIMD
        sink = torch.empty(blocks * 256, dtype=torch.float32, device=dev)
        flops = blocks * 4 * args.issue_probe_iters * 4 * 32768.0
        res = {}
        for name, mix in (("mfma_only_tflops", False), ("with_sweep_mix_tflops", True)):
            B.issue_probe(mix, blocks, args.issue_probe_iters, sink)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(5):
                B.issue_probe(mix, blocks, args.issue_probe_iters, sink)
            e1.record(stream)
            e1.synchronize()
            res[name] = round(flops / (e0.elapsed_time(e1) * 1e-3 / 5) / 1e12, 1)
        res["mix_share"] = round(res["with_sweep_mix_tflops"] / res["mfma_only_tflops"], 4)
        issue = res
        del sink

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    assert int(cu_ret[-1].item()) == out_rows
    if args.copy_probe_mib > 0:  # one plain copy of known size, for counter calibration
        n = args.copy_probe_mib << 20
        src_buf = torch.ones(n, dtype=torch.uint8, device=dev)
        dst_buf = torch.empty_like(src_buf)
        dst_buf.copy_(src_buf)
        torch.cuda.synchronize()
        del src_buf, dst_buf

    stage_names = (["score", "select", "compact"] if shared
                   else ["saliency", "priority", "select", "compact"])
    if args.decode:
        stage_names.append("decode")
    # the timed pass: K steps with no event inside a step (an event record leaves the
    # GPU idle for about 5 us); then the same K steps again with a HIP event around each
    # C ABI call, for the per-stage times and the roofline of the saliency stage
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for i in range(args.steps):
        step()
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_end)
    ms_per_step = max(total_ms, wall * 1e3) / args.steps

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stage_names) + 1)]
           for _ in range(args.steps)]
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    stage_ms = {n: float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs]))
                for i, n in enumerate(stage_names)}


    tokens = float(ntot)
    value = tokens / (ms_per_step * 1e-3)
    G = w.num_q_heads // Hkv
    R = w.window * G
    lh = L * Hkv
    # algorithmic work per launch of the saliency stage (in shared mode: the
    # scoring call, whose sweeps cover the last n layers only)
    sweeps = 1 if args.lse_fed else 2
    lh_sal = (n_sh * Hkv) if shared else lh
    k_bytes = lh_sal * ntot * d * 2
    sal_flops = sweeps * 2 * R * d * ntot * lh_sal     # Q K^T once per sweep
    sal_bytes = k_bytes + lh_sal * ntot * 4 + q.numel() * 2 * lh_sal // lh  # K, A, Q
    if args.lse_fed:
        sal_bytes += lse.numel() * 4 * lh_sal // lh
    compact_bytes = lh * out_rows * d * 2 * 2 * 2     # K and V rows, read and written
    t_sal = stage_ms["score" if shared else "saliency"] * 1e-3
    t_cmp = stage_ms["compact"] * 1e-3
    achieved_tflops = sal_flops / t_sal / 1e12
    achieved_gbs = sal_bytes / t_sal / 1e9
    kernel = ("saliency (one MFMA sweep over K, row LSE given)" if args.lse_fed
              else "saliency (two MFMA sweeps over K)")
    if shared:
        kernel = f"shared-index scoring: {kernel} of the last {n_sh} layers, head sum, priority"
    traffic = recorded_traffic(traffic_key(args.workload, budget, w.window, args.lse_fed,
                                           n_sh if shared else 0, args.schedule))
    # the binding roofline: whichever of HBM and MFMA needs longer at peak
    if sal_bytes / (HBM_PEAK_GBS * 1e9) >= sal_flops / (BF16_PEAK_TFLOPS * 1e12):
        roofline = {"bound": "hbm", "achieved": round(achieved_gbs, 1), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(achieved_gbs / HBM_PEAK_GBS, 4)}
    else:
        roofline = {"bound": "mfma", "achieved": round(achieved_tflops, 2),
                    "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(achieved_tflops / BF16_PEAK_TFLOPS, 4)}
    roofline.update({"traffic": traffic, "kernel": kernel})
    hbm = {"saliency_gbps": round(sal_bytes / t_sal / 1e9, 1),
           "saliency_frac": round(sal_bytes / t_sal / 1e9 / HBM_PEAK_GBS, 4),
           "compact_gbps": round(compact_bytes / t_cmp / 1e9, 1),
           "compact_frac": round(compact_bytes / t_cmp / 1e9 / HBM_PEAK_GBS, 4),
           "peak_gbps": HBM_PEAK_GBS}
    if traffic:  # the counted bytes of the saliency stage over its time
        hbm.update({"saliency_measured_gbps": round(traffic / t_sal / 1e9, 1),
                    "saliency_measured_frac": round(traffic / t_sal / 1e9 / HBM_PEAK_GBS, 4)})
    if args.decode:  # K_hat and V_hat read once (plus queries and outputs)
        dec_bytes = lh * out_rows * d * 2 * 2 + q_dec.numel() * 2 + dec_out.numel() * 4
        t_dec = stage_ms["decode"] * 1e-3
        hbm.update({"decode_gbps": round(dec_bytes / t_dec / 1e9, 1),
                    "decode_frac": round(dec_bytes / t_dec / 1e9 / HBM_PEAK_GBS, 4)})

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {L} layers, {w.num_q_heads} query / {Hkv} KV "
                               f"heads, d {d}, {w.num_seqs} sequence(s) of {w.seqlens[:4]}"
                               f"{'...' if w.num_seqs > 4 else ''} tokens, window {w.window}, "
                               f"budget {budget} per KV head"
                               + (", row LSE given" if args.lse_fed else "")
                               + (", causal window" if args.causal_tail else "")
                               + (f", one ranking per sequence from the last {n_sh} layers"
                                  if shared else "")
                               + (", step signals from text" if args.text_signals else "")
                               + (f", {args.selector} selector" if args.selector != "stepkv"
                                  else ""),
                   "selector": args.selector,
                   "text_signals": bool(args.text_signals),
                   "shared_layers": n_sh if shared else 0,
                   "saliency_sweeps": sweeps, "saliency_schedule": args.schedule,
                   "causal_tail": bool(args.causal_tail),
                   "layers": L, "kv_heads": Hkv, "q_heads": w.num_q_heads, "head_dim": d,
                   "seq_len": int(max(w.seqlens)), "tokens": int(ntot), "window": w.window,
                   "budget": budget, "seed": args.seed},
        "entries_per_s": round(value * lh, 1),
        "stages_ms": {n: round(x, 4) for n, x in stage_ms.items()},
        "hbm": hbm,
        "roofline": roofline,
    }
    if flushed:
        line["flushed"] = flushed
    if ceilings:
        line["hbm_ceilings"] = ceilings
    if issue:
        line["mfma_issue"] = issue
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = (cpu_baseline_shared(w, budget, args.cpu_seconds, params, n_sh)
                                if shared else
                                cpu_baseline(w, budget, args.cpu_seconds, params, args.lse_fed))
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
