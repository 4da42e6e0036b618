#!/usr/bin/env python3
"""Benchmark of one decode step of HillInfer's token-importance path on one
MI355X: for every layer, score all cached keys against the step's query and
update the cumulative importance, select the top-k tokens, and attend over
them (libhill ``hill_step_streamed``: the selection takes the previous step's
threshold as a running bound, Sec. 4.2 HIE; results identical to
``hill_step``, which is timed beside it).

Default workload: the Llama-3-8B-shaped 32K-context decode -- 32 layers, GQA
32 query / 8 KV heads, head_dim 128, batch 1, 32768 cached bf16 tokens per
layer, keys with LogNormal(0,1) per-channel outlier scales, budget 10%
(3276 tokens), importance carried across the decode steps.  A "step" is one
decode step through all 32 layers.  Inputs are synthetic (seeded), resident
in HBM before timing starts; the 4 GiB of K+V exceed the 256 MB Infinity
Cache, so every layer's keys come from HBM.

Prints one JSON line:
  value        scoring GB/s: the keys of one layer (B*Hkv*n*D*2 bytes) over
               the scoring stage of one layer-step (the key scan plus the
               normaliser and S update), with each stage's duration taken from
               start/stop timestamps that its own dispatch stamps into HIP
               events (one probe layer per step, on the library's stream)
  ms_per_step  wall time of one decode step through all layers (timed region
               bracketed by device synchronisations)
  roofline     the key-scan kernel (score_tiles): algorithmic bytes per
               launch / its mean duration (the scan stage's events) vs 8 TB/s
  stage_us     mean duration per stage of a layer-step (scan, update,
               select, merge; refine in the plain leg)
  select_attn_us_per_layer_step   select + merge stages (selection, gather,
               attention over the selected tokens, merge of the partials),
               beside dense_decode_bound_us, the time to read all K and V of
               a layer once at 8 TB/s
  plain        the same steps through hill_step (refine pass, five launches)
  bkp          the hot/cold pool pass after each layer's step (Sec. 4.2 BKP)
  sketch, sketch4  the same steps scored on the int8 / int4 key sketch
               (Sec. 4.4 asymmetric precision): step time, scan roofline on
               its own bytes, selection agreement with the 16-bit path
  tier         the tiered cache (hot pool of 2k rows in HBM, the rest in
               pinned host memory read in place) on 4 layers: stage times
               beside the int8 sketch leg's, the BKP pass and the row
               migration per layer, the share of selected rows in the hot pool
  kernel_traffic  calibrated HBM bytes per launch of update_attn, topk_emit
               and merge_write beside their algorithmic bytes (committed
               counter runs; null once their sources changed)
  cpu_baseline the CPU oracle on a bounded sample of the same workload

Other modes: ``--sweep`` (27-cell throughput sweep, one line per cell),
``--copy-calib`` (plain copy of known size, for counter calibration),
``--read-ceiling`` (a plain streaming read at the scan's sizes),
``--selection-stats`` (heavy-hitter recall of the Qwen-7B-shaped workload and
the step-to-step selection overlap of the AR(1) workload),
``--summarize DIR`` (condense rocprofv3 output under DIR into text), ``--summarize-sweep DIR`` (per-cell kernel
medians of a rocprofv3 kernel trace of ``--sweep``),
``--counters DIR`` (score_tiles HBM traffic from rocprofv3 --pmc runs),
``--step-counters DIR`` (the same for update_attn, topk_emit, merge_write).
"""
from __future__ import annotations

import argparse
import ctypes
import dataclasses
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "scoring GB/s of K scanned (% HBM peak) + select+attn µs/layer-step at 32K ctx"
COUNTERS_FILE = os.path.join(ROOT, "profiles", "score_tiles_counters.json")
SCORE_SRC = os.path.join(ROOT, "paper_2602_18750_amd", "csrc", "score.hip")
COUNTERS_WORKLOAD = 3   # the counters are taken on the default workload (Llama-3-8B-shaped 32K)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ------------------------------------------------------------- HIP events --

class StageProbe:
    """Start/stop events for every stage of one decode step (include/hill.h
    HILL_STAGE_*), and the stage durations they measured.  The events are
    torch's (HIP events with timing, created by a first record on the
    stream), so that they belong to the HIP runtime that torch and the
    library share; their handles go to the library, which stamps them at the
    start and end of each stage's launch."""

    def __init__(self, H, stream):
        import torch
        self.stages = H.hill.STAGES
        self.start = [torch.cuda.Event(enable_timing=True) for _ in self.stages]
        self.stop = [torch.cuda.Event(enable_timing=True) for _ in self.stages]
        for e in self.start + self.stop:
            e.record(stream)
        self.ev = H.HillStepEvents.of([e.cuda_event for e in self.start], [e.cuda_event for e in self.stop])

    def us(self, stage: str) -> float:
        i = self.stages.index(stage)
        return self.start[i].elapsed_time(self.stop[i]) * 1e3


def stage_means(probes, stages):
    """Mean duration (us) of each named stage over the probes."""
    return {st: sum(p.us(st) for p in probes) / len(probes) for st in stages}


# ------------------------------------------------------------ byte counts --

def scan_kernel_bytes(B, Hq, Hkv, D, n, mode="attn"):
    """Algorithmic bytes of one score_tiles launch: every key read once, plus
    (ATTN) the fp32 logits and the per-256-token (max, sum) pairs of every
    head written (an even number of pairs per head)."""
    kbytes = B * Hkv * n * D * 2
    if mode != "attn":
        return kbytes + B * n * 4 * 2
    units = (n + 255) // 256
    npart = (units + 1) // 2 * 2
    return kbytes + B * Hq * n * 4 + B * Hq * npart * 8


def load_traffic(which="keys16"):
    """HBM traffic of one score_tiles launch (which = "keys16" for the scan of
    the 16-bit keys, "sketch" / "sketch4" for the scan of the int8 / int4
    sketch) from committed counter runs, only while the kernel source is
    unchanged since the counters were taken."""
    try:
        rec = json.load(open(COUNTERS_FILE))
        src = hashlib.sha256(open(SCORE_SRC, "rb").read()).hexdigest()
        if rec.get("source_sha256") != src:
            return None
        if which in ("sketch", "sketch4"):
            return (rec.get(which) or {}).get("hbm_bytes_per_launch")
        return rec.get("hbm_bytes_per_launch")
    except (OSError, ValueError):
        return None


# ------------------------------------------------------------- CPU oracle --

def cpu_baseline(w, seconds: float):
    """The oracle, as it stands, on a bounded sample: consecutive decode steps
    of layer 0 of the same workload (full context), S carried."""
    import numpy as np
    import torch
    from oracle import oracle as O
    from paper_2602_18750_amd import workloads as W

    x = W.make_layer(w.replace(steps=max(2, min(w.steps, 64))), 0)

    def u16(t):
        return t.contiguous().view(torch.int16).numpy().view(np.uint16)

    kb, vb = u16(x.k), u16(x.v)
    R = 1
    S = np.zeros((w.batch, R, w.n_tokens))
    done, t_total, phases = 0, 0.0, np.zeros(3)
    while done < x.q.shape[0]:
        t0 = time.perf_counter()
        S, _, _, ph = O.step(u16(x.q[done]), kb, vb, S, w.k_sel, w.dtype, "attn", "token", return_times=True)
        t_total += time.perf_counter() - t0
        phases += ph
        done += 1
        if t_total >= seconds and done >= 2:
            break
    kbytes = w.batch * w.n_kv_heads * w.n_tokens * w.head_dim * 2
    per = t_total / done
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {
        "value": round(kbytes / per / 1e9, 4),
        "unit": "GB/s",
        "cores": O.num_threads(),
        "affinity_cpus": len(os.sched_getaffinity(0)),
        "cpu_model": model,
        "kind": "oracle",
        "sample": "%d decode steps of layer 0 (B=%d, n=%d, GQA %d/%d, %s, k=%d), S carried; "
                  "%.1f ms per layer-step (score %.1f, select %.1f, attention %.1f)" % (
                      done, w.batch, w.n_tokens, w.n_q_heads, w.n_kv_heads, w.dtype, w.k_sel, per * 1e3,
                      phases[0] / done * 1e3, phases[1] / done * 1e3, phases[2] / done * 1e3),
    }


# ------------------------------------------------------------- main bench --

def run_bench(args):
    import torch
    import paper_2602_18750_amd as H
    from paper_2602_18750_amd import workloads as W

    w = W.WORKLOADS[int(args.workload)]
    if args.layers:
        w = w.replace(layers=args.layers)
    if args.n_tokens:
        w = w.replace(n_tokens=args.n_tokens, name="%s-n%d" % (w.name, args.n_tokens))
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    nl, T = w.layers, w.steps
    log("bench: %s, %d layers, %d query steps, k=%d" % (w.name, nl, T, w.k_sel))

    layers = []
    for L in range(nl):
        x = W.make_layer(w, L, device=dev)
        s = H.new_importance(w.batch, 1, w.n_tokens, dev)
        layers.append((x, s))
    # workloads smaller than 1 GiB of K+V would stay in the 256 MB Infinity
    # Cache across steps: their layers are replicated (fresh copies of K and V,
    # own S) and the step walks all replicas, so keys come from HBM as in a
    # real model; per-step figures are normalised back to one pass of nl layers
    kv_bytes = 2 * nl * w.batch * w.n_kv_heads * w.n_tokens * w.head_dim * 2
    reps = max(1, min(16, -(-(1 << 30) // kv_bytes)))
    for r in range(1, reps):
        for L in range(nl):
            x = layers[L][0]
            xr = dataclasses.replace(x, k=x.k.clone(), v=x.v.clone())
            layers.append((xr, H.new_importance(w.batch, 1, w.n_tokens, dev)))
    nl_run = nl * reps
    ws = H.workspace(H.make_desc(layers[0][0].q[0], layers[0][0].k, layers[0][0].v, layers[0][1]), w.k_sel, dev)
    states = [H.new_stream_state(w.batch, 1, dev) for _ in layers]   # one running bound per S buffer
    calls = [H.StepCall(x.q[0], x.k, x.v, s, w.k_sel, ws=ws, stream=stream, stream_state=states[L])
             for L, (x, s) in enumerate(layers)]
    qptrs = [[x.q[t].data_ptr() for t in range(T)] for (x, _) in layers]
    torch.cuda.synchronize()

    probes = [StageProbe(H, stream) for _ in range(args.steps)]

    for i in range(args.warmup):
        for L in range(nl_run):
            calls[L](qptrs[L][i % T])
    torch.cuda.synchronize()

    t0 = time.perf_counter()
    for i in range(args.steps):
        t = (args.warmup + i) % T
        probe = i % nl_run        # one timestamped layer per step, rotating
        for L in range(nl_run):
            if L == probe:
                calls[L](qptrs[L][t], probes[i].ev)
            else:
                calls[L](qptrs[L][t])
    torch.cuda.synchronize()
    t1 = time.perf_counter()

    st = stage_means(probes, ("scan", "update", "select", "merge"))

    ms_step = (t1 - t0) * 1e3 / (args.steps * reps)   # one decode step = nl layer-steps
    kbytes_layer = w.batch * w.n_kv_heads * w.n_tokens * w.head_dim * 2
    vbytes_layer = kbytes_layer
    scan_bytes = scan_kernel_bytes(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.n_tokens)
    scan_us = st["scan"]
    achieved = scan_bytes / (scan_us * 1e-6) / 1e9
    score_us = st["scan"] + st["update"]
    scoring_gbs = kbytes_layer / (score_us * 1e-6) / 1e9
    traffic = load_traffic() if w.id == COUNTERS_WORKLOAD else None

    res = {
        "metric": METRIC,
        "value": round(scoring_gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "batch": w.batch, "n_q_heads": w.n_q_heads, "n_kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
            "n_tokens": w.n_tokens, "budget": w.budget, "k_sel": w.k_sel, "layers": nl,
            "query_steps": T, "score_mode": "attn", "granularity": "token", "selection": "streamed",
            "parallelism": "none (1 GPU)",
            "kv_replicas": reps,
        },
        "roofline": {
            "kernel": "score_tiles",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": scan_bytes,
            "mean_launch_us": round(scan_us, 3),
        },
        "scoring_frac_hbm": round(scoring_gbs / HBM_PEAK_GBS, 4),
        "scoring_us_per_layer_step": round(score_us, 3),
        "select_attn_us_per_layer_step": round(st["select"] + st["merge"], 3),
        "dense_decode_bound_us": round((kbytes_layer + vbytes_layer) / (HBM_PEAK_GBS * 1e3), 3),
        "stage_us": {k: round(v, 3) for k, v in st.items()},
        "layer_step_us_wall": round(ms_step * 1e3 / nl, 3),
        "step_keys_gbps": round(kbytes_layer * nl / (ms_step * 1e-3) / 1e9, 1),
    }
    if w.id == COUNTERS_WORKLOAD:
        res["kernel_traffic"] = load_step_traffic()
    if not args.no_plain:
        res["plain"] = bench_plain(args, w, layers, nl, nl_run, reps, T, qptrs, ws, stream)
    if not args.no_bkp:
        res["bkp"] = bench_bkp(args, w, calls, nl_run, T, qptrs, stream)
    if not args.no_sketch:
        res["sketch"] = bench_sketch(args, w, layers, nl, nl_run, reps, T, qptrs, ws, stream, 8)
        res["sketch4"] = bench_sketch(args, w, layers, nl, nl_run, reps, T, qptrs, ws, stream, 4)
    if not args.no_tier:
        res["tier"] = bench_tier(args, w, layers, T, qptrs, ws, stream)
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle (%.0f s budget)" % args.cpu_seconds)
        res["cpu_baseline"] = cpu_baseline(W.WORKLOADS[int(args.workload)], args.cpu_seconds)
    else:
        res["cpu_baseline"] = None
    print(json.dumps(res), flush=True)


def bench_plain(args, w, layers, nl, nl_run, reps, T, qptrs, ws, stream):
    """The same decode steps through hill_step (the selection's refine pass,
    five launches per layer-step), fresh S per layer."""
    import torch
    import paper_2602_18750_amd as H

    dev = torch.device("cuda:0")
    ss = [H.new_importance(w.batch, 1, w.n_tokens, dev) for _ in layers]
    calls = [H.StepCall(x.q[0], x.k, x.v, ss[L], w.k_sel, ws=ws, stream=stream) for L, (x, _) in enumerate(layers)]
    probes = [StageProbe(H, stream) for _ in range(args.steps)]
    for i in range(args.warmup):
        for L in range(nl_run):
            calls[L](qptrs[L][i % T])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        t = (args.warmup + i) % T
        probe = i % nl_run
        for L in range(nl_run):
            if L == probe:
                calls[L](qptrs[L][t], probes[i].ev)
            else:
                calls[L](qptrs[L][t])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    st = stage_means(probes, ("scan", "update", "refine", "select", "merge"))
    ms_step = (t1 - t0) * 1e3 / (args.steps * reps)
    del calls, ss
    return {
        "ms_per_step": round(ms_step, 4),
        "step_keys_gbps": round(w.batch * w.n_kv_heads * w.n_tokens * w.head_dim * 2 * nl / (ms_step * 1e-3) / 1e9,
                                1),
        "scoring_us_per_layer_step": round(st["scan"] + st["update"], 3),
        "select_attn_us_per_layer_step": round(st["refine"] + st["select"] + st["merge"], 3),
        "stage_us": {k: round(v, 3) for k, v in st.items()},
        "launches_per_layer_step": 5,
    }


def bench_bkp(args, w, calls, nl_run, T, qptrs, stream):
    """The Bidirectional KV Cache Pools pass (Sec. 4.2 BKP) after each
    layer's decode step, on that step's selected set: recent window = k
    tokens (alpha * N), hot pool = 2k tokens (the window plus the top-alpha
    by hit count).  Timed per pass with events around one probe layer per
    step; the decode steps themselves run untimed in between."""
    import torch
    import paper_2602_18750_amd as H

    dev = torch.device("cuda:0")
    k = w.k_sel
    states = [H.BkpState(w.batch, 1, w.n_tokens, dev) for _ in range(nl_run)]
    bkps = [H.BkpCall(st, k, n_tokens=w.n_tokens, n_recent=k, capacity=2 * k, stream=stream) for st in states]
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for i in range(args.steps):
        t = i % T
        probe = i % nl_run
        for L in range(nl_run):
            calls[L](qptrs[L][t])
            if L == probe:
                evs[i][0].record(stream)
            bkps[L](calls[L].idx.data_ptr())
            if L == probe:
                evs[i][1].record(stream)
    torch.cuda.synchronize()
    us = sorted(a.elapsed_time(b) * 1e3 for a, b in evs[1:])   # the first pass fills the empty pools
    last = bkps[(args.steps - 1) % nl_run].counts[0, 0].tolist()
    del bkps, states
    return {
        "us_per_pass_median": round(us[len(us) // 2], 3),
        "us_per_pass_mean": round(sum(us) / len(us), 3),
        "n_recent": k, "capacity": 2 * k, "launches_per_pass": 6,
        "last_pass_promotions": last[0], "last_pass_demotions": last[1],
    }


def bench_tier(args, w, layers, T, qptrs, ws, stream, n_layers=4):
    """The tiered KV cache (Sec. 4.2 BKP with the rows moved): per layer a hot
    pool of 2k slot rows in HBM and the cold rows in pinned host memory that
    the attention reads in place; after each layer's decode step the BKP pass
    over its selection and the migration of the rows it names.  The step
    scores on the int8 sketch, so its stages compare with the int8 sketch
    leg's (all rows in HBM).  ``n_layers`` layers, one probe layer per step
    (stage events on its step, events around its BKP pass and its
    migration); the first 8 steps fill the pools and stay untimed."""
    import torch
    import paper_2602_18750_amd as H

    dev = torch.device("cuda:0")
    k = w.k_sel
    nt = min(n_layers, len(layers))
    caches = [H.TieredCache(layers[L][0].k, layers[L][0].v, 2 * k, bits=8, stream=stream) for L in range(nt)]
    ss = [H.new_importance(w.batch, 1, w.n_tokens, dev) for _ in range(nt)]
    sts = [H.new_stream_state(w.batch, 1, dev) for _ in range(nt)]
    steps = [H.TierStepCall(layers[L][0].q[0], caches[L], ss[L], k, n_tokens=w.n_tokens, ws=ws, stream=stream,
                            stream_state=sts[L]) for L in range(nt)]
    bstates = [H.BkpState(w.batch, 1, w.n_tokens, dev) for _ in range(nt)]
    bkps = [H.BkpCall(b, k, n_tokens=w.n_tokens, n_recent=k, capacity=2 * k, stream=stream) for b in bstates]
    moves = [H.TierApplyCall(caches[L], bkps[L], n_tokens=w.n_tokens, stream=stream) for L in range(nt)]
    fill = 8
    n_steps = max(args.steps, nt)
    probes = [StageProbe(H, stream) for _ in range(n_steps)]
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_steps)]
    snap = None
    torch.cuda.synchronize()
    t0 = None
    for i in range(fill + n_steps):
        if i == fill:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
        t = i % T
        j = i - fill
        probe = j % nt if j >= 0 else -1
        for L in range(nt):
            if L == probe:
                steps[L](qptrs[L][t], probes[j].ev)
                if j == n_steps - 1:     # the last probe step's selection and where its rows were
                    snap = (L, steps[L].idx.clone(), caches[L].loc.clone())
                ev[j][0].record(stream)
                bkps[L](steps[L].idx.data_ptr())
                ev[j][1].record(stream)
                moves[L]()
                ev[j][2].record(stream)
            else:
                steps[L](qptrs[L][t])
                bkps[L](steps[L].idx.data_ptr())
                moves[L]()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    st = stage_means(probes, ("scan", "update", "select", "merge"))
    bkp_us = sorted(a.elapsed_time(b) * 1e3 for a, b, _ in ev)
    mig_us = sorted(b.elapsed_time(c) * 1e3 for _, b, c in ev)
    sel, loc = snap[1].long().clamp_min(0), snap[2]
    in_hot = float((loc.gather(2, sel) >= 0).float().mean())
    status = int(caches[0].status.item())
    hot_rows = [int((c.loc[0, 0] >= 0).sum()) for c in caches]
    row_bytes = 2 * w.n_kv_heads * w.head_dim * 2    # K and V of one token
    counts = bkps[0].counts[0, 0].tolist()
    del steps, moves, bkps, caches
    torch.cuda.empty_cache()
    return {
        "layers": nt,
        "capacity": 2 * k, "n_recent": k, "granularity": "token",
        "layer_step_us_wall": round((t1 - t0) * 1e6 / (n_steps * nt), 3),
        "stage_us": {kk: round(v, 3) for kk, v in st.items()},
        "select_attn_us_per_layer_step": round(st["select"] + st["merge"], 3),
        "bkp_pass_us_median": round(bkp_us[len(bkp_us) // 2], 3),
        "migration_us_median": round(mig_us[len(mig_us) // 2], 3),
        "migration_us_mean": round(sum(mig_us) / len(mig_us), 3),
        "last_pass_promotions": counts[0], "last_pass_demotions": counts[1],
        "moved_bytes_last_pass": (counts[0] + counts[1]) * row_bytes,
        "hot_rows": hot_rows,
        "selected_in_hot_pool": round(in_hot, 4),
        "status": status,
    }


def bench_sketch(args, w, layers, nl, nl_run, reps, T, qptrs, ws, stream, nbits=8):
    """The same decode steps scored on the int8 (nbits 8) or int4 (nbits 4)
    key sketch (Sec. 4.4 asymmetric precision; the streamed selection and the
    attention as in the main leg).  The sketches are written once before timing, as when the
    cache is filled; in a decode loop only the appended row is sketched per
    step."""
    import torch
    import paper_2602_18750_amd as H

    dev = torch.device("cuda:0")
    sks = [H.sketch_keys(x.k, bits=nbits) for (x, _) in layers]
    ss = [H.new_importance(w.batch, 1, w.n_tokens, dev) for _ in layers]
    states = [H.new_stream_state(w.batch, 1, dev) for _ in layers]
    calls = [H.StepCall(x.q[0], x.k, x.v, ss[L], w.k_sel, ws=ws, stream=stream, sketch=sks[L],
                        stream_state=states[L]) for L, (x, _) in enumerate(layers)]
    probes = [StageProbe(H, stream) for _ in range(args.steps)]
    for i in range(args.warmup):
        for L in range(nl_run):
            calls[L](qptrs[L][i % T])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        t = (args.warmup + i) % T
        probe = i % nl_run
        for L in range(nl_run):
            if L == probe:
                calls[L](qptrs[L][t], probes[i].ev)
            else:
                calls[L](qptrs[L][t])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    st = stage_means(probes, ("scan", "update", "select", "merge"))
    scan = st["scan"] * 1e-3                     # ms
    score = (st["scan"] + st["update"]) * 1e-3
    selattn = (st["select"] + st["merge"]) * 1e-3
    ms_step = (t1 - t0) * 1e3 / (args.steps * reps)
    units = (w.n_tokens + 255) // 256
    npart = (units + 1) // 2 * 2
    scan_bytes = (w.batch * w.n_kv_heads * w.n_tokens * (128 * nbits // 8 + 1)
                  + w.batch * w.n_q_heads * w.n_tokens * 4 + w.batch * w.n_q_heads * npart * 8)
    scan_gbs = scan_bytes / (scan * 1e-3) / 1e9
    traffic = load_traffic("sketch" if nbits == 8 else "sketch4")
    # selection agreement with the 16-bit path: one step from zero importance on layer 0
    x = layers[0][0]
    s16 = H.new_importance(w.batch, 1, w.n_tokens, dev)
    s8 = H.new_importance(w.batch, 1, w.n_tokens, dev)
    i16, _ = H.hill_step(x.q[0], x.k, x.v, s16, w.k_sel, ws=ws, stream=stream)
    i8, _ = H.hill_step(x.q[0], x.k, x.v, s8, w.k_sel, ws=ws, stream=stream, sketch=sks[0])
    torch.cuda.synchronize()
    a, b = i16.cpu(), i8.cpu()
    recall = sum(len(set(a[r, 0].tolist()) & set(b[r, 0].tolist())) for r in range(w.batch)) / (w.batch * w.k_sel)
    del calls, sks, ss, states
    return {
        "ms_per_step": round(ms_step, 4),
        "value_gbps_of_16bit_keys": round(w.batch * w.n_kv_heads * w.n_tokens * w.head_dim * 2 * nl /
                                          (ms_step * 1e-3) / 1e9, 2),
        "scan_us": round(scan * 1e3, 3),
        "scan_algorithmic_bytes": scan_bytes,
        "scan_gbps": round(scan_gbs, 1),
        "scan_frac_hbm": round(scan_gbs / HBM_PEAK_GBS, 4),
        "scan_traffic": traffic if w.id == COUNTERS_WORKLOAD else None,
        "scoring_us_per_layer_step": round(score * 1e3, 3),
        "select_attn_us_per_layer_step": round(selattn * 1e3, 3),
        "stage_us": {k: round(v, 3) for k, v in st.items()},
        "selection_recall_vs_16bit": round(recall, 4),
    }


# ------------------------------------------------------------------ sweep --

def run_sweep(args):
    """Throughput sweep: one decode step per cell, K rotated through enough
    replicas to exceed 1 GiB so that the scan reads HBM, not the Infinity Cache."""
    import torch
    import paper_2602_18750_amd as H
    from paper_2602_18750_amd import workloads as W

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    for w in W.sweep_workloads():
        kv_bytes = 2 * w.batch * w.n_kv_heads * w.n_tokens * w.head_dim * 2
        reps = max(1, min(16, -(-(1 << 30) // kv_bytes)))
        x = W.make_layer(w, 0, device=dev, seed=7000)
        ks = [x.k] + [x.k.clone() for _ in range(reps - 1)]
        vs = [x.v] + [x.v.clone() for _ in range(reps - 1)]
        s = H.new_importance(w.batch, 1, w.n_tokens, dev)
        ws = H.workspace(H.make_desc(x.q[0], x.k, x.v, s), w.k_sel, dev)
        calls = [H.StepCall(x.q[0], ks[r], vs[r], s, w.k_sel, ws=ws, stream=stream) for r in range(reps)]
        iters = max(20, reps)
        probes = [StageProbe(H, stream) for _ in range(iters)]
        for r in range(reps):
            calls[r](x.q[0].data_ptr())
        torch.cuda.synchronize()
        for i in range(iters):
            calls[i % reps](x.q[0].data_ptr(), probes[i].ev)
        torch.cuda.synchronize()

        def med(f):
            return sorted(f(p) for p in probes)[iters // 2] * 1e-3   # ms
        scan = med(lambda p: p.us("scan"))
        score = med(lambda p: p.us("scan") + p.us("update"))
        selattn = med(lambda p: p.us("refine") + p.us("select") + p.us("merge"))
        nbytes = scan_kernel_bytes(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.n_tokens)
        kbytes = w.batch * w.n_kv_heads * w.n_tokens * w.head_dim * 2
        print(json.dumps({
            "cell": w.name, "batch": w.batch, "n_tokens": w.n_tokens, "budget": w.budget, "k_sel": w.k_sel,
            "scan_us": round(scan * 1e3, 2), "scan_gbps": round(nbytes / (scan * 1e-3) / 1e9, 1),
            "scan_frac_hbm": round(nbytes / (scan * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "scoring_us": round(score * 1e3, 2),
            "scoring_kgbps": round(kbytes / (score * 1e-3) / 1e9, 1),
            "select_attn_us": round(selattn * 1e3, 2), "replicas": reps}), flush=True)
        del calls, ks, vs, x, s, probes
        torch.cuda.empty_cache()


def run_selection_stats(args):
    """Statistics of the selections the path makes (not pass/fail; the GPU
    tests hold the same figures against the oracle):
    * Qwen-7B-shaped workload (32 layers, B 8, 4096 tokens, 5% heavy-hitter
      keys scaled 4x): the fraction of heavy-hitter tokens inside the selected
      set of one decode step, per layer and overall;
    * the AR(1) workload (B 4, 131072 tokens, 16 decode steps, streamed
      selection as in the benchmark): the overlap |I_t & I_(t-1)| / k of
      consecutive selections per step (temporal locality, Sec. 4.2)."""
    import torch
    import paper_2602_18750_amd as H
    from paper_2602_18750_amd import workloads as W

    dev = torch.device("cuda:0")
    w = W.WORKLOADS[2]
    recalls = []
    for L in range(w.layers):
        x = W.make_layer(w, L, device=dev)
        s = H.new_importance(w.batch, 1, w.n_tokens, dev)
        idx, _ = H.hill_step(x.q[0], x.k, x.v, s, w.k_sel)
        torch.cuda.synchronize()
        hv = x.heavy.to(dev).long()
        chosen = torch.zeros(w.batch, w.n_tokens, dtype=torch.bool, device=dev)
        chosen.scatter_(1, idx[:, 0].long(), True)
        recalls.append(float(torch.gather(chosen, 1, hv).float().mean()))
        del x, s, idx
    print(json.dumps({"workload": w.name, "statistic": "heavy-hitter recall in the selected set",
                      "k_sel": w.k_sel, "heavy_per_row": int(W.HEAVY_FRACTION * w.n_tokens),
                      "per_layer": [round(r, 4) for r in recalls],
                      "mean": round(sum(recalls) / len(recalls), 4), "min": round(min(recalls), 4)}), flush=True)

    w = W.WORKLOADS[4]
    x = W.make_layer(w, 0, device=dev)
    s = H.new_importance(w.batch, 1, w.n_tokens, dev)
    state = H.new_stream_state(w.batch, 1, dev)
    call = H.StepCall(x.q[0], x.k, x.v, s, w.k_sel, stream_state=state)
    prev, overlap = None, []
    for t in range(w.steps):
        call(x.q[t].data_ptr())
        torch.cuda.synchronize()
        cur = torch.zeros(w.batch, w.n_tokens, dtype=torch.bool, device=dev)
        cur.scatter_(1, call.idx[:, 0].long(), True)
        if prev is not None:
            overlap.append(float((cur & prev).sum(1).float().mean()) / w.k_sel)
        prev = cur
    print(json.dumps({"workload": w.name, "statistic": "overlap |I_t & I_(t-1)| / k of consecutive selections",
                      "k_sel": w.k_sel, "steps": w.steps, "per_step": [round(o, 4) for o in overlap],
                      "mean": round(sum(overlap) / len(overlap), 4)}), flush=True)


def run_copy_calib(args):
    """A plain elementwise copy of known size (counter calibration): 1 GiB
    read and 1 GiB written by one kernel (bitwise_not of uint8), three times.
    FETCH_SIZE and WRITE_SIZE of these dispatches against their known bytes
    give the factors that turn the counters into HBM bytes."""
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda:0")
    b = torch.empty(n, dtype=torch.uint8, device="cuda:0")
    a.fill_(1)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.bitwise_not(a, out=b)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n, "repeats": 3}), flush=True)


def run_read_ceiling(args):
    """What a single plain streaming-read launch reaches at the scan's sizes:
    the calibration read (libhill_calib.so hill_calib_read: 16-byte non-temporal
    loads, eight in flight per lane, one contiguous share per workgroup) over
    16 MiB .. 1 GiB, the best of a few grid sizes, rotated through replicas so
    that at least 1 GiB is touched between reuses; event-timed like the scan."""
    import torch
    from paper_2602_18750_amd import _build
    lib = ctypes.CDLL(_build.CALIB_LIB)
    lib.hill_calib_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    lib.hill_calib_read.restype = ctypes.c_int

    def calib_read(buf, grid, sink, stream):
        rc = lib.hill_calib_read(buf.data_ptr(), buf.numel(), grid, sink.data_ptr(), stream.cuda_stream)
        if rc != 0:
            raise RuntimeError("hill_calib_read failed (%d)" % rc)

    stream = torch.cuda.current_stream()
    sink = torch.empty(65536, dtype=torch.int32, device="cuda:0")
    for mib in (16, 32, 64, 256, 1024):
        reps = max(1, min(16, 1024 // mib))
        xs = [torch.empty(mib << 20, dtype=torch.uint8, device="cuda:0").fill_(r + 1) for r in range(reps)]
        best = None
        per_grid = {}
        for grid in (1024, 2048, 4096, 8192):
            for x in xs:
                calib_read(x, grid, sink, stream)
            torch.cuda.synchronize()
            iters = max(20, reps)
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters)]
            for i in range(iters):
                ev[i][0].record(stream)
                calib_read(xs[i % reps], grid, sink, stream)
                ev[i][1].record(stream)
            torch.cuda.synchronize()
            ts = sorted(a.elapsed_time(b) for a, b in ev)
            med = ts[len(ts) // 2]
            per_grid[grid] = round(med * 1e3, 2)
            if best is None or med < best[0]:
                best = (med, grid)
        med, grid = best
        gbs = (mib << 20) / (med * 1e-3) / 1e9
        print(json.dumps({"read_mib": mib, "kernel": "hill_calib_read", "grid": grid, "median_us": round(med * 1e3, 2),
                          "gbps": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 4), "replicas": reps,
                          "median_us_per_grid": per_grid}),
              flush=True)
        del xs
        torch.cuda.empty_cache()


def _counter_rows(directory: str, counter: str, name_part: str, steady: bool = False):
    """Per-dispatch values of `counter` for kernels whose name contains
    name_part (a regular expression); with `steady`, only the later half of
    the dispatches in launch order (the bench's timed steps after as many
    warm-up steps, which hold the reset steps of every fresh S)."""
    import csv
    vals = []
    for path in sorted(glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True)):
        with open(path) as f:
            per = {}
            for r in csv.DictReader(f):
                if r.get("Counter_Name") != counter or not re.search(name_part, r.get("Kernel_Name", "")):
                    continue
                key = int(r.get("Dispatch_Id") or r.get("Correlation_Id"))
                per[key] = per.get(key, 0.0) + float(r.get("Counter_Value", 0))
            xs = [per[k] for k in sorted(per)]
            vals.extend(xs[len(xs) // 2:] if steady else xs)
    return vals


STEP_SOURCES = [os.path.join(ROOT, "paper_2602_18750_amd", "csrc", f)
                for f in ("update.hip", "topk.hip", "attn_device.h", "hill_device.h", "hill_internal.h")]
STEP_COUNTERS_FILE = os.path.join(ROOT, "profiles", "step_kernels_counters.json")


def step_sources_sha() -> str:
    h = hashlib.sha256()
    for p in STEP_SOURCES:
        h.update(open(p, "rb").read())
    return h.hexdigest()


def step_algorithmic_bytes(B, Hq, Hkv, D, n, k):
    """Algorithmic bytes per launch of the streamed step's kernels after the
    scan (token rows, ATTN weights, 16-bit V; 512-token selection chunks,
    128-token update blocks, 256-token scan units):
      update_attn  the logits (Hq * 4 B per token), the scan's unit partials
                   once, S read and written (the candidate pairs, 8 B each
                   for the few thousand tokens at or above the bound's bin,
                   and the sparse histogram bins are left out)
      topk_emit    the selected tokens' V rows, the G heads' logits of every
                   chunk (at a 5-20 % budget every 128-byte line of them holds
                   selected tokens), S, and the (m, l, o) partials written
      merge_write  the partials, the chunk lists and the index output, the
                   output rows."""
    nchunks = -(-n // 512)
    npart = (-(-n // 256) + 1) // 2 * 2
    parts = B * Hq * nchunks * (D + 2) * 4
    return {
        "update_attn": B * Hq * n * 4 + B * Hq * npart * 8 + 2 * B * n * 4,
        "topk_emit": B * k * Hkv * D * 2 + B * Hq * n * 4 + B * n * 4 + parts,
        "merge_write": parts + 2 * B * k * 4 + B * Hq * D * 4,
    }


def make_step_counters(directory: str, command: str):
    """The HBM-traffic record of the streamed step's kernels after the scan
    (update_attn, topk_emit streamed with the scan's logits, merge_write) at
    workload 3, from the same four --pmc runs as make_counters (steady-state
    dispatches only), with each kernel's algorithmic bytes and the ratio."""
    from paper_2602_18750_amd import workloads as W

    def mean(xs):
        if not xs:
            raise SystemExit("no dispatches found under %s" % directory)
        return sum(xs) / len(xs)

    copy_bytes = 1 << 30
    ff = copy_bytes / (mean(_counter_rows(os.path.join(directory, "calib_fetch"), "FETCH_SIZE", "bitwise_not")) * 1024.0)
    wf = copy_bytes / (mean(_counter_rows(os.path.join(directory, "calib_write"), "WRITE_SIZE", "bitwise_not")) * 1024.0)
    w = W.WORKLOADS[COUNTERS_WORKLOAD]
    alg = step_algorithmic_bytes(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.n_tokens, w.k_sel)
    names = {"update_attn": r"update_attn_kernel",
             "topk_emit": r"topk_emit_kernel<1, 4, true, true, true, false>",
             "merge_write": r"merge_write_kernel"}
    rec = {"workload": w.name, "source_sha256": step_sources_sha(), "fetch_factor": round(ff, 4),
           "write_factor": round(wf, 4), "kernels": {}, "command": command}
    for key, pat in names.items():
        fs = _counter_rows(os.path.join(directory, "fetch"), "FETCH_SIZE", pat, steady=True)
        ws_ = _counter_rows(os.path.join(directory, "write"), "WRITE_SIZE", pat, steady=True)
        hbm = mean(fs) * 1024.0 * ff + mean(ws_) * 1024.0 * wf
        rec["kernels"][key] = {"dispatches": len(fs), "fetch_kib_per_dispatch": round(mean(fs), 1),
                               "write_kib_per_dispatch": round(mean(ws_), 1), "hbm_bytes_per_launch": int(round(hbm)),
                               "algorithmic_bytes_per_launch": alg[key], "traffic_over_algorithmic": round(hbm / alg[key], 3)}
    print(json.dumps(rec, indent=1))


def load_step_traffic():
    """The step kernels' traffic record, while their sources are unchanged."""
    try:
        rec = json.load(open(STEP_COUNTERS_FILE))
        return rec["kernels"] if rec.get("source_sha256") == step_sources_sha() else None
    except (OSError, ValueError, KeyError):
        return None


def make_counters(directory: str, command: str):
    """Writes the score_tiles HBM-traffic record from four rocprofv3 --pmc runs
    under `directory`: fetch/ and write/ (FETCH_SIZE, WRITE_SIZE of the bench),
    calib_fetch/ and calib_write/ (the same counters of --copy-calib)."""
    def mean(xs):
        if not xs:
            raise SystemExit("no dispatches found under %s" % directory)
        return sum(xs) / len(xs)

    copy_bytes = 1 << 30
    cf_kib = mean(_counter_rows(os.path.join(directory, "calib_fetch"), "FETCH_SIZE", "bitwise_not"))
    cw_kib = mean(_counter_rows(os.path.join(directory, "calib_write"), "WRITE_SIZE", "bitwise_not"))
    ff = copy_bytes / (cf_kib * 1024.0)
    wf = copy_bytes / (cw_kib * 1024.0)

    def scan(keys):   # the score_tiles instantiations matching `keys` (a regular expression)
        f_kib = mean(_counter_rows(os.path.join(directory, "fetch"), "FETCH_SIZE", keys))
        w_kib = mean(_counter_rows(os.path.join(directory, "write"), "WRITE_SIZE", keys))
        return {"fetch_kib_per_dispatch": round(f_kib, 1), "write_kib_per_dispatch": round(w_kib, 1),
                "hbm_bytes_per_launch": int(round(f_kib * 1024.0 * ff + w_kib * 1024.0 * wf))}

    rec = {"kernel": "score_tiles (16-bit keys)",
           "source_sha256": hashlib.sha256(open(SCORE_SRC, "rb").read()).hexdigest()}
    rec.update(scan(r"KeysF16"))
    rec.update({
        "copy_bytes": copy_bytes,
        "copy_fetch_kib": round(cf_kib, 1),
        "copy_write_kib": round(cw_kib, 1),
        "fetch_factor": round(ff, 4),
        "write_factor": round(wf, 4),
        "sketch": dict(kernel="score_tiles (int8 key sketch)", **scan(r"KeysSketchMfma8<|KeysSketch<\d+, \d+, 8>")),
        "sketch4": dict(kernel="score_tiles (int4 key sketch)", **scan(r"KeysSketchMfma4<|KeysSketch<\d+, \d+, 4>")),
        "command": command,
    })
    print(json.dumps(rec, indent=1))


# -------------------------------------------------------- profile summary --

def _short(name: str) -> str:
    name = name.replace("(anonymous namespace)::", "").replace("void ", "")
    depth, out = 0, []
    for ch in name:            # drop the argument list, keep template arguments
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    return "".join(out)[:80]


def _steady_state(path: str, directory: str):
    """Median durations of the streamed decode step's four kernels (scan over
    the 16-bit keys, update, streamed select+attend, merge), taken from the
    launches in that order in a kernel trace, without the first third of them
    (the first steps of every fresh S run without a bound)."""
    import csv
    import statistics
    with open(path) as f:
        rows = sorted(csv.DictReader(f), key=lambda r: int(r["Start_Timestamp"]))
    names = [_short(r["Kernel_Name"]) for r in rows]
    seqs, i = [], 0
    while i + 3 < len(rows):
        n = names[i:i + 4]
        if (n[0].startswith("hill::score_tiles_kernel") and "KeysF16" in n[0] and n[1] == "hill::update_attn_kernel"
                and n[2].startswith("hill::topk_emit_kernel") and n[2].count("true") >= 2
                and n[3] == "hill::merge_write_kernel"):
            seqs.append(rows[i:i + 4])
            i += 4
        else:
            i += 1
    if not seqs:
        return []
    steady = seqs[len(seqs) // 3:]
    out = ["## %s: streamed decode step, steady state" % os.path.relpath(path, directory),
           "%d layer-steps in the trace, the last %d used (median µs per launch)" % (len(seqs), len(steady)),
           "", "| kernel | median us |", "|---|---|"]
    for k in range(4):
        d = [(int(sq[k]["End_Timestamp"]) - int(sq[k]["Start_Timestamp"])) / 1e3 for sq in steady]
        out.append("| %s | %.2f |" % (_short(steady[0][k]["Kernel_Name"]), statistics.median(d)))
    return out


def summarize(directory: str):
    """Condense rocprofv3 --stats / --pmc CSV output found under `directory`."""
    import csv
    lines = []
    for path in sorted(glob.glob(os.path.join(directory, "**", "*kernel_stats.csv"), recursive=True)):
        lines.append("## %s" % os.path.relpath(path, directory))
        lines.append("| kernel | calls | mean us | total % |")
        lines.append("|---|---|---|---|")
        with open(path) as f:
            for r in csv.DictReader(f):
                short = _short(r.get("Name", ""))
                lines.append("| %s | %s | %.3f | %.2f |" % (short, r.get("Calls"), float(r.get("AverageNs", 0)) / 1e3,
                                                          float(r.get("Percentage", 0))))
    for path in sorted(glob.glob(os.path.join(directory, "**", "*kernel_trace.csv"), recursive=True)):
        lines.extend(_steady_state(path, directory))
    for path in sorted(glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True)):
        agg = {}
        with open(path) as f:
            for r in csv.DictReader(f):
                name = _short(r.get("Kernel_Name", ""))
                key = (name, r.get("Counter_Name"))
                agg.setdefault(key, []).append(float(r.get("Counter_Value", 0)))
        lines.append("## %s" % os.path.relpath(path, directory))
        lines.append("| kernel | counter | dispatches | mean per dispatch |")
        lines.append("|---|---|---|---|")
        for (name, ctr), vals in sorted(agg.items()):
            lines.append("| %s | %s | %d | %.1f |" % (name, ctr, len(vals), sum(vals) / len(vals)))
    print("\n".join(lines))


def summarize_sweep(directory: str):
    """Per-cell kernel durations of `bench.py --sweep` from a rocprofv3 kernel
    trace under `directory`: the sweep's cells run in workloads.sweep_workloads()
    order, each as `replicas` warm-up steps and max(20, replicas) timed steps of
    hill_step (scan, update, refine, select+attend, merge); per cell the median
    duration of each kernel over the timed steps, and the scan's roofline
    fraction (its algorithmic bytes over that median, against 8 TB/s)."""
    import csv
    import statistics
    from paper_2602_18750_amd import workloads as W

    path = sorted(glob.glob(os.path.join(directory, "**", "*kernel_trace.csv"), recursive=True))
    if not path:
        raise SystemExit("no kernel trace under %s" % directory)
    with open(path[0]) as f:
        rows = sorted(csv.DictReader(f), key=lambda r: int(r["Start_Timestamp"]))
    kinds = (("scan", "score_tiles_kernel"), ("stats", "softmax_stats_kernel"), ("update", "update_attn_kernel"),
             ("refine", "topk_refine_kernel"), ("select", "topk_emit_kernel"), ("merge", "merge_write_kernel"))
    # one step per scan launch: the kernels up to the next scan belong to it
    # (softmax_stats runs only where the update does not reduce the partials)
    steps = []
    for r in rows:
        for k, pat in kinds:
            if pat in r["Kernel_Name"]:
                if k == "scan":
                    steps.append({})
                elif not steps:
                    raise SystemExit("trace starts with a %s launch before any scan" % k)
                steps[-1][k] = steps[-1].get(k, 0.0) + (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3
                break
    pos = 0
    out = ["| cell (B, n, α) | k | scan µs | scan GB/s | frac of 8 TB/s | stats µs | update µs | refine µs | select µs | "
           "merge µs | step µs |",
           "|---|---|---|---|---|---|---|---|---|---|---|"]
    for w in W.sweep_workloads():
        kv_bytes = 2 * w.batch * w.n_kv_heads * w.n_tokens * w.head_dim * 2
        reps = max(1, min(16, -(-(1 << 30) // kv_bytes)))
        iters = max(20, reps)
        cell = steps[pos + reps:pos + reps + iters]
        pos += reps + iters
        if len(cell) != iters:
            raise SystemExit("trace holds fewer steps than the sweep makes")
        med = {k: statistics.median(st.get(k, 0.0) for st in cell) for k, _ in kinds}
        nbytes = scan_kernel_bytes(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.n_tokens)
        gbs = nbytes / (med["scan"] * 1e-6) / 1e9
        out.append("| %d, %dK, %d%% | %d | %.2f | %.0f | %.3f | %.2f | %.2f | %.2f | %.2f | %.2f | %.2f |" % (
            w.batch, w.n_tokens // 1024, round(w.budget * 100), w.k_sel, med["scan"], gbs, gbs / HBM_PEAK_GBS,
            med["stats"], med["update"], med["refine"], med["select"], med["merge"], sum(med.values())))
    print("\n".join(out))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="3", help="1..4 (default 3: the 32K-context Llama-3-8B-shaped decode)")
    ap.add_argument("--layers", type=int, default=None)
    ap.add_argument("--n-tokens", type=int, default=None, help="context length override (a variant of the workload)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sketch", action="store_true", help="skip the int8 / int4 sketch variants of the step")
    ap.add_argument("--no-tier", action="store_true", help="skip the tiered-cache leg (hot pool in HBM, cold in host)")
    ap.add_argument("--no-bkp", action="store_true", help="skip timing the hot/cold pool pass")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--sweep", action="store_true")
    ap.add_argument("--copy-calib", action="store_true")
    ap.add_argument("--read-ceiling", action="store_true", help="time a plain streaming read at the scan's sizes")
    ap.add_argument("--selection-stats", action="store_true",
                    help="heavy-hitter recall (Qwen-7B-shaped) and step-to-step selection overlap (AR(1) workload)")
    ap.add_argument("--summarize", metavar="DIR")
    ap.add_argument("--summarize-sweep", metavar="DIR", help="per-cell kernel medians of a rocprofv3 trace of --sweep")
    ap.add_argument("--counters", metavar="DIR", help="write the score_tiles traffic record from --pmc runs under DIR")
    ap.add_argument("--step-counters", metavar="DIR",
                    help="write the traffic record of the step's other kernels from --pmc runs under DIR")
    ap.add_argument("--counters-command", default="", help="command line recorded with --counters")
    ap.add_argument("--no-plain", action="store_true", help="skip the hill_step (refine pass) leg")
    args = ap.parse_args()

    if args.counters:
        make_counters(args.counters, args.counters_command)
        return 0
    if args.step_counters:
        make_step_counters(args.step_counters, args.counters_command)
        return 0

    if args.summarize:
        summarize(args.summarize)
        return 0
    if args.summarize_sweep:
        summarize_sweep(args.summarize_sweep)
        return 0
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this path has no multi-GPU mode "
              "(--gpus %d, WORLD_SIZE %d requested)" % (args.gpus, world), file=sys.stderr)
        return 2
    if args.copy_calib:
        run_copy_calib(args)
    elif args.read_ceiling:
        run_read_ceiling(args)
    elif args.selection_stats:
        run_selection_stats(args)
    elif args.sweep:
        run_sweep(args)
    else:
        run_bench(args)
    return 0


if __name__ == "__main__":
    sys.exit(main())
