#!/usr/bin/env python3
"""Throughput of the HedgeSpec drafter-evaluation hot path on one MI355X.

A step is one verification round of the whole path on one batch of synthetic logits:
temperature softmax statistics, alpha = sum min(p, q_i) for every drafter and position,
Theorem 3's expected acceptance length, the length loss, and the Hedge and NormalHedge
updates (hs_round: one launch of the evaluation kernel, which folds the slice sums into alpha
and runs each query's learner step once its alpha is complete).

Default workload: the large drafter pool (B=32 queries, N=64 drafters, K=8 positions,
V=151936, bf16 logits, T=1, Hedge with eta = sqrt(8 ln N / 1000) and NormalHedge), the largest
configuration, 5.06 GB of logits per round. Inputs are resident in HBM before timing starts;
successive steps rotate through distinct rounds (at least two, and >= 512 MB in all) so that
the 256 MB Infinity Cache cannot serve a repeated input. Steps run as HIP graph replays; every
graph is captured before the timed region.

Prints one JSON line. `value` = drafter-positions evaluated per second (B*N*K per step).
`roofline` prices one hs_eval_alpha call (one launch of the team kernel, timed with HIP events
on the stream it runs on, over calls replayed back to back) against HBM bandwidth with
algorithmic bytes (every logit read once); `traffic` is the counter-measured HBM bytes of that
call from the committed FETCH_SIZE / WRITE_SIZE summary of the workload, null if there is
none or the kernel sources changed since it was taken. `cpu_baseline` times the float64 oracle
on the host, on all cores and on one thread.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
ROTATE_BYTES = 512 * 1024 * 1024
METRIC = "drafter-positions evaluated/sec + achieved HBM GB/s (% of peak), 1 MI355X"
# Sources of the evaluation kernels; a counter summary is valid only for these bytes.
KERNEL_SOURCES = ["paper_2510_20064_amd/csrc/hs_team.hip", "paper_2510_20064_amd/csrc/hs_wave.h",
                  "paper_2510_20064_amd/csrc/hs_internal.h", "paper_2510_20064_amd/csrc/hs_learner.h"]


def kernel_source_digest() -> str:
    import hashlib

    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def pmc_summary_path(name: str) -> str:
    return os.path.join(ROOT, "profiles", "hs_eval_alpha_%s_pmc.md" % name)


def measured_traffic(name: str):
    """HBM bytes per hs_eval_alpha call from the committed FETCH_SIZE / WRITE_SIZE summary of
    this workload, or None when there is none or the kernel sources changed since."""
    path = pmc_summary_path(name)
    if not os.path.exists(path):
        return None
    rec = None
    with open(path) as f:
        for ln in f:
            if ln.startswith("traffic-record: "):
                rec = json.loads(ln[len("traffic-record: "):])
    if not rec or rec.get("kernel_sources_sha256") != kernel_source_digest():
        return None
    return rec["hbm_bytes_per_call"]


TOPL_SOURCES = ["paper_2510_20064_amd/csrc/hs_topl.hip", "paper_2510_20064_amd/csrc/hs_wave.h",
                "paper_2510_20064_amd/csrc/hs_internal.h"]


def measured_topl_traffic(workload: str):
    """HBM bytes per hs_eval_topl call (both launches) from the committed counter summary of this
    workload, or None when there is none or the kernel sources changed since it was taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", "hs_eval_topl_%s.md" % workload)
    if not os.path.exists(path):
        return None
    rec = None
    with open(path) as f:
        for ln in f:
            if ln.startswith("traffic-record: "):
                rec = json.loads(ln[len("traffic-record: "):])
    h = hashlib.sha256()
    for rel in TOPL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    if not rec or rec.get("kernel_sources_sha256") != h.hexdigest():
        return None
    return rec["hbm_bytes_per_call"]


LOGIT_TYPES = ("fp32", "bf16", "fp16")  # by the library's dtype code (HS_F32, HS_BF16, HS_F16)


def logit_type(w) -> str:
    return LOGIT_TYPES[w.dtype]


def profile_name(w, name: str) -> str:
    """The counter summary that covers this run (the workloads' own storage types have one)."""
    return name + "_f16" if LOGIT_TYPES[w.dtype] == "fp16" and not name.endswith("_f16") else name


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="large_pool_stream")
    ap.add_argument("--stack", type=int, default=1, metavar="R",
                    help="R independent instances of the workload per step (R times the "
                         "queries, each with its own logits; for the latency-bound small shapes)")
    ap.add_argument("--cpu-seconds", type=float, default=18.0,
                    help="approximate CPU time budget of the oracle baseline, two thirds on all "
                         "cores and one third on one thread (0 = skip)")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--pruned", type=float, default=0.0, metavar="KEEP",
                    help="with --topl: also time hs_candidate_mass on the children pruned to "
                         "a seeded KEEP fraction (Theorem 2 with dynamic pruning)")
    ap.add_argument("--f16", action="store_true",
                    help="store the workload's logits as fp16 (IEEE binary16) instead")
    ap.add_argument("--greedy", action="store_true",
                    help="evaluate in greedy argmax-agreement mode (the workload's second run)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--read-calibration", action="store_true",
                    help="also time hs_stream_read, a plain streaming read of the resident "
                         "inputs: this device's achievable read rate")
    ap.add_argument("--topl", type=int, default=0, metavar="L",
                    help="time hs_eval_topl (EAGLE's top-L acceptance mass, Theorem 2) with L "
                         "children per node on the workload instead")
    ap.add_argument("--hybrid", type=int, default=0, metavar="H",
                    help="with --delayed: the acceptance loss for each query's first H tokens")
    ap.add_argument("--bookkeeping", action="store_true",
                    help="time one round of drafter play (argmax of NormalHedge's p) and regret "
                         "bookkeeping (hs_play + hs_regret_update) on the workload's B, N")
    ap.add_argument("--softmax-stats", action="store_true",
                    help="time hs_softmax_stats over every row of the workload instead")
    ap.add_argument("--delayed", action="store_true",
                    help="time hs_delayed_update (token-level delayed feedback) on the workload's "
                         "B, N, K instead, K new tokens per query per round")
    return ap.parse_args()


def bench_delayed(args, w, hs, torch, dev):
    """hs_delayed_update in steady state: every call brings K new tokens per query, so each
    query's learners take K window losses in order (K NormalHedge solves per query)."""
    B, N, K = w.B, w.N, w.K
    copies = 16
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed)
    gam = [torch.rand((B, N, K), generator=gen, device=dev) for _ in range(copies)]
    cnt = torch.full((B,), K, dtype=torch.int32, device=dev)
    st = hs.DelayedState(B, N, K, dev)
    stream = torch.cuda.Stream()

    def call(i):
        hs.delayed_update(st, gam[i % copies], cnt, w.eta, hybrid_tokens=args.hybrid,
                          stream=torch.cuda.current_stream())

    with torch.cuda.stream(stream):
        for i in range(copies):  # past the first K tokens: every later call completes K windows
            call(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for i in range(copies):
            call(i)
    torch.cuda.synchronize()
    reps = max(1, args.steps // copies)
    with torch.cuda.stream(stream):
        for _ in range(max(1, args.warmup // copies)):
            g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    with torch.cuda.stream(stream):
        for _ in range(reps):
            g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (reps * copies)
    nl = st.nloss.cpu()
    assert bool(torch.all(nl == K)), "steady state expected K windows per query per call"
    # bytes a call moves: gamma in, history ring in and out, learner state in and out, losses out
    nbytes = B * N * K * 4 + 2 * B * 2 * K * N * 4 + 2 * 5 * B * N * 8 + B * K * N * 8
    line = {"metric": "delayed-feedback learner: drafter-window losses used per second",
            "value": B * N * K / (us * 1e-6), "unit": "drafter-windows/s", "n_gpus": 1,
            "steps": reps * copies, "warmup": max(1, args.warmup // copies) * copies,
            "us_per_call": us, "higher_is_better": True, "dtype": "f64", "data": "synthetic",
            "config": {"workload": w.name, "B": B, "N": N, "K": K, "eta": w.eta,
                       "tokens_per_call": K, "hybrid_tokens": args.hybrid, "hip_graph": True},
            "roofline": {"bound": "latency", "achieved": nbytes / (us * 1e-6) / 1e9,
                         "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                         "kernel": "hs_delayed_kernel (one wave per query, K sequential window "
                                   "updates each)", "bytes_per_call": nbytes}}
    print(json.dumps(line), flush=True)


def bench_bookkeeping(args, w, hs, torch, dev):
    """One round of play and bookkeeping: hs_play (argmax of NormalHedge's p) and
    hs_regret_update with the round's loss vector, in a HIP graph."""
    B, N = w.B, w.N
    copies = 16
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed)
    p = torch.rand((B, N), generator=gen, device=dev, dtype=torch.float64)
    loss = [torch.rand((1, B, N), generator=gen, device=dev, dtype=torch.float64)
            for _ in range(copies)]
    eal = torch.rand((B, N), generator=gen, device=dev, dtype=torch.float64) * (w.K + 1)
    choice = torch.empty((B,), dtype=torch.int32, device=dev)
    reg = hs.RegretState(B, N, dev)
    stream = torch.cuda.Stream()

    def call(i):
        cs = torch.cuda.current_stream()
        hs.play(p, hs.PLAY_ARGMAX, out=choice, stream=cs)
        reg.update(loss[i % copies], choice.view(1, B), eal, stream=cs)

    with torch.cuda.stream(stream):
        for i in range(copies):
            call(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for i in range(copies):
            call(i)
    torch.cuda.synchronize()
    reps = max(1, args.steps // copies)
    with torch.cuda.stream(stream):
        for _ in range(max(1, args.warmup // copies)):
            g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    with torch.cuda.stream(stream):
        for _ in range(reps):
            g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (reps * copies)
    nbytes = B * N * 8 * 5 + B * 4 * 2 + B * 8 * 4  # p, loss, eal, cum in/out; choice; sums
    line = {"metric": "drafter play and regret bookkeeping: rounds per second",
            "value": 1.0 / (us * 1e-6), "unit": "rounds/s", "n_gpus": 1, "steps": reps * copies,
            "warmup": max(1, args.warmup // copies) * copies, "us_per_call": us,
            "higher_is_better": True, "dtype": "f64", "data": "synthetic",
            "config": {"workload": w.name, "B": B, "N": N, "play": "argmax", "hip_graph": True},
            "roofline": {"bound": "latency", "achieved": nbytes / (us * 1e-6) / 1e9,
                         "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                         "kernel": "hs_play_kernel + hs_regret_kernel (one wave per query each)",
                         "bytes_per_call": nbytes}}
    print(json.dumps(line), flush=True)


def bench_softmax_stats(args, w, hs, torch, dev, synth):
    """hs_softmax_stats over every row of the workload (target and drafters, all queries and
    positions) on distinct rounds resident in HBM (>= 512 MB, rotated), in a HIP graph. The
    roofline prices a call at each logit read once plus the three outputs per row."""
    copies = max(1, math.ceil(ROTATE_BYTES / w.input_bytes))
    if w.input_bytes * copies > 64e9:
        copies = max(1, int(64e9 // w.input_bytes))
    bufs = []
    for r in range(copies):
        x = synth.generate(w, round=r)
        t = torch.from_numpy(x.reshape(-1, x.shape[-1]))
        if w.dtype == synth.BF16:
            t = t.view(torch.bfloat16)
        bufs.append(t.to(dev))
        del x, t
    rows = bufs[0].shape[0]
    out = (torch.empty(rows, dtype=torch.float32, device=dev),
           torch.empty(rows, dtype=torch.float32, device=dev),
           torch.empty(rows, dtype=torch.int32, device=dev))
    stream = torch.cuda.Stream()

    def call(i):
        hs.softmax_stats(bufs[i % copies], V=w.V, temperature=w.temperature, out=out,
                         stream=torch.cuda.current_stream())

    with torch.cuda.stream(stream):
        for i in range(copies):
            call(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for i in range(copies):
            call(i)
    torch.cuda.synchronize()
    reps = max(1, args.steps // copies)
    with torch.cuda.stream(stream):
        for _ in range(max(1, args.warmup // copies)):
            g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    with torch.cuda.stream(stream):
        for _ in range(reps):
            g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (reps * copies)
    if args.copy_calibration:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    nbytes = rows * w.V * w.elem_bytes + rows * 12
    achieved = nbytes / (us * 1e-6) / 1e9
    line = {"metric": "softmax row statistics: rows per second + achieved HBM GB/s",
            "value": rows / (us * 1e-6), "unit": "rows/s", "n_gpus": 1,
            "steps": reps * copies, "warmup": max(1, args.warmup // copies) * copies,
            "us_per_call": us, "higher_is_better": True, "dtype": "f32", "data": "synthetic",
            "config": {"workload": w.name, "rows": rows, "V": w.V,
                       "logits": logit_type(w),
                       "temperature": w.temperature, "rotation_copies": copies,
                       "hip_graph": True},
            "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                         "kernel": "hs_softmax_stats (one workgroup per row)",
                         "bytes_per_call": nbytes}}
    print(json.dumps(line), flush=True)


def bench_pruned(args, w, hs, torch, np, bufs, copies, L):
    """hs_candidate_mass after hs_eval_topl: each copy's children with a seeded (1 - KEEP)
    share of the slots emptied, the target's lse from hs_softmax_stats; graph-replayed calls
    over the resident copies, timed with HIP events."""
    T = w.temperature
    rng = np.random.default_rng(12)
    lses, cands, outs = [], [], []
    for i in range(copies):
        o = hs.eval_topl(bufs[i], L=L, V=w.V, temperature=T, want_gamma=True, want_hit=False,
                         want_children=True)
        c = o["children"].cpu().numpy()
        c[rng.random(c.shape) >= args.pruned] = -1
        cands.append(torch.from_numpy(c).cuda())
        tgt = bufs[i][0]
        _, lse, _ = hs.softmax_stats(tgt.reshape(w.B * w.K, -1), V=w.V, temperature=T)
        lses.append(lse.reshape(w.B, w.K))
        outs.append(torch.empty((w.B, w.N, w.K), dtype=torch.float32, device=tgt.device))
    stream = torch.cuda.Stream()

    def call(i):
        hs.candidate_mass(bufs[i][0], lses[i], cands[i], V=w.V, temperature=T, out=outs[i],
                          stream=torch.cuda.current_stream())

    per_graph = max(copies, 16)  # a short kernel: several calls per replay amortise its launch
    with torch.cuda.stream(stream):
        for i in range(copies):
            call(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for i in range(per_graph):
            call(i % copies)
    torch.cuda.synchronize()
    reps = max(1, args.steps // per_graph)
    with torch.cuda.stream(stream):
        for _ in range(max(1, args.warmup // per_graph)):
            g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    with torch.cuda.stream(stream):
        for _ in range(reps):
            g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (reps * per_graph)
    kept = float(np.mean([(c >= 0).float().mean().item() for c in cands]))
    outputs = w.B * w.N * w.K
    # bytes a call needs: the candidate lists, one lse per group, the kept target logits, gamma
    nbytes = outputs * L * 4 + w.B * w.K * 4 + outputs * L * kept * w.elem_bytes + outputs * 4
    return {"kernel": "hs_candidate_mass (one launch)", "us_per_call": us,
            "outputs_per_s": outputs / (us * 1e-6), "keep_fraction": round(kept, 4),
            "slots_per_output": L, "bytes_per_call": int(nbytes),
            "achieved_GBps": nbytes / (us * 1e-6) / 1e9, "bound": "latency"}


def bench_topl(args, w, hs, torch, dev, np, synth):
    """hs_eval_topl on distinct rounds resident in HBM (>= 512 MB, rotated), in a HIP graph.
    A call is two launches (per-slice candidates, then the merge); the roofline prices the whole
    call against every logit read once."""
    L = args.topl
    copies = max(1, math.ceil(ROTATE_BYTES / w.input_bytes))
    if w.input_bytes * copies > 64e9:
        copies = max(1, int(64e9 // w.input_bytes))
    bufs = []
    for r in range(copies):
        t = torch.from_numpy(synth.generate(w, round=r))
        if w.dtype == synth.BF16:
            t = t.view(torch.bfloat16)
        bufs.append(t.to(dev))
    ws = torch.empty(hs.topl_workspace_size(w.B, w.N, w.K, w.V, L, w.dtype), dtype=torch.uint8,
                     device=dev)
    greedy = w.mode == hs.GREEDY
    out = {}
    stream = torch.cuda.Stream()

    def call(i):
        hs.eval_topl(bufs[i % copies], L=L, V=w.V, temperature=w.temperature, mode=w.mode,
                     workspace=ws, out=out, stream=torch.cuda.current_stream())

    with torch.cuda.stream(stream):
        for i in range(copies):
            call(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for i in range(copies):
            call(i)
    torch.cuda.synchronize()
    reps = max(1, args.steps // copies)
    with torch.cuda.stream(stream):
        for _ in range(max(1, args.warmup // copies)):
            g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    with torch.cuda.stream(stream):
        for _ in range(reps):
            g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    us = e0.elapsed_time(e1) * 1e3 / (reps * copies)
    achieved = w.input_bytes / (us * 1e-6) / 1e9
    pruned = bench_pruned(args, w, hs, torch, np, bufs, copies, L) if args.pruned > 0 else None
    if args.copy_calibration:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()

    cpu = None
    if args.cpu_seconds > 0:
        import oracle

        x = synth.generate(w, round=0)
        t1 = time.perf_counter()
        n_done = 0
        G = w.B * w.K
        xg = x.reshape(x.shape[0], G, x.shape[-1])
        while True:  # one (query, position) group at a time: all N drafters of it
            gi = n_done % G
            oracle.topl(xg[:, gi:gi + 1], L, V=w.V, T=w.temperature, want_mass=not greedy)
            n_done += 1
            el = time.perf_counter() - t1
            if el >= args.cpu_seconds:
                break
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        threads = min(threads, os.cpu_count() or threads)
        cpu = {"value": w.N * n_done / el, "unit": "drafter-positions/s", "cores": threads,
               "kind": "oracle",
               "sample": "%d (query, position) groups of the same workload, all %d drafters each, "
                         "float64 C oracle (L passes per row) with OpenMP over rows, %.1f s"
                         % (n_done, w.N, el)}
    line = {"metric": "EAGLE top-L acceptance mass: " + METRIC,
            "value": w.positions / (us * 1e-6), "unit": "drafter-positions/s", "n_gpus": 1,
            "steps": reps * copies, "warmup": max(1, args.warmup // copies) * copies,
            "ms_per_step": us * 1e-3, "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "i32 keys, f32 mass", "data": "synthetic",
            "config": {"workload": w.name, "B": w.B, "N": w.N, "K": w.K, "V": w.V, "L": L,
                       "logits": logit_type(w),
                       "temperature": w.temperature, "mode": "greedy" if greedy else "sample",
                       "rotation_copies": copies, "input_bytes_per_step": w.input_bytes,
                       "hip_graph": True, "wall_s": round(wall, 4)},
            "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                         "traffic": measured_topl_traffic(profile_name(w, w.name)),
                         "kernel": "hs_eval_topl = hs_topl_slice_kernel + hs_topl_merge_kernel "
                                   "(one call, both launches timed)",
                         "kernel_us": us, "algorithmic_bytes_per_launch": w.input_bytes},
            "cpu_baseline": cpu}
    if pruned:
        line["pruned_mass"] = pruned
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one MI355X: the library has no multi-GPU path "
              "(queries would shard across GPUs with no exchange between them). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2510_20064_amd as hs
    import synth

    hs.load_library()
    w = synth.workloads()[args.workload]
    if args.greedy:
        w = synth.variant(w, mode=synth.GREEDY)
    if args.stack > 1:  # R independent instances: R times the queries, each its own logits
        w = synth.variant(w, B=w.B * args.stack)
    if args.f16:
        w = synth.variant(w, dtype=synth.F16)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.delayed:
        bench_delayed(args, w, hs, torch, dev)
        return
    if args.topl:
        bench_topl(args, w, hs, torch, dev, np, synth)
        return
    if args.bookkeeping:
        bench_bookkeeping(args, w, hs, torch, dev)
        return
    if args.softmax_stats:
        bench_softmax_stats(args, w, hs, torch, dev, synth)
        return

    # ---- inputs: distinct rounds, resident in HBM -----------------------------------------
    copies = max(2, math.ceil(ROTATE_BYTES / w.input_bytes))
    if w.input_bytes * copies > 64e9:
        copies = max(1, int(64e9 // w.input_bytes))
    bufs = []
    for r in range(copies):
        x = synth.generate(w, round=r)
        t = torch.from_numpy(x)
        if w.dtype == synth.BF16:
            t = t.view(torch.bfloat16)
        bufs.append(t.to(dev))
        del x, t
    parent = w.parent()
    path_end = w.path_end()
    pe_dev = None if path_end is None else torch.from_numpy(path_end).to(dev)

    rounds = []
    state = hs.LearnerState(w.B, w.N, dev)
    for r in range(copies):
        rounds.append(hs.Round(bufs[r], V=w.V, temperature=w.temperature, mode=w.mode,
                               loss_kind=w.loss, eta=w.eta, parent=parent, path_end=pe_dev,
                               state=state, want_loss=False))
    torch.cuda.synchronize()

    stream = torch.cuda.Stream()
    greedy = w.mode == hs.GREEDY
    use_graph = not args.no_graph

    def step_fn(i):
        rounds[i % copies].run(stream=torch.cuda.current_stream())

    ev_ws = hs.alloc_workspace(w.B, w.N, w.K, w.V, w.dtype, dev)
    ev_out = ({"agree": torch.empty((w.B, w.N, w.K), dtype=torch.uint8, device=dev)} if greedy
              else {"alpha": torch.empty((w.B, w.N, w.K), dtype=torch.float32, device=dev)})

    def eval_fn(i):
        hs.eval_alpha(bufs[i % copies], V=w.V, temperature=w.temperature, mode=w.mode,
                      workspace=ev_ws, out=ev_out, stream=torch.cuda.current_stream())

    # ---- every graph the timed regions replay, captured up front ----------------------------
    graphs = {}

    def capture(fn, n):
        key = (fn.__name__, n)
        if n == 0 or key in graphs:
            return
        with torch.cuda.stream(stream):
            for i in range(n):  # one eager pass before capture
                fn(i)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for i in range(n):
                fn(i)
        torch.cuda.synchronize()
        graphs[key] = g

    def run(fn, n):
        """n calls of fn (in rounds of `copies`), replaying graphs captured beforehand."""
        if not use_graph:
            with torch.cuda.stream(stream):
                for i in range(n):
                    fn(i)
            return
        full, rem = divmod(n, copies)
        with torch.cuda.stream(stream):
            for _ in range(full):
                graphs[(fn.__name__, copies)].replay()
            if rem:
                graphs[(fn.__name__, rem)].replay()

    n_eval = copies * max(1, args.steps // copies)
    if use_graph:
        for n in {copies, args.steps % copies, args.warmup % copies}:
            capture(step_fn, n)
        capture(eval_fn, copies)

    # ---- warmup + timed region: the hs_round steps ------------------------------------------
    run(step_fn, args.warmup)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    run(step_fn, args.steps)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = e0.elapsed_time(e1) / args.steps
    value = w.positions / (ms_step * 1e-3)

    # ---- the whole 1000-round stream of the large pool (hs_round per round, the learners
    # carried through), inputs rotating as above ------------------------------------------------
    stream_total = None
    if w.name == "large_pool_stream" and args.stack == 1 and use_graph:
        rounds_total = 1000
        capture(step_fn, rounds_total % copies)  # (every other graph exists already)
        torch.cuda.synchronize()
        e6 = torch.cuda.Event(enable_timing=True)
        e7 = torch.cuda.Event(enable_timing=True)
        e6.record(stream)
        run(step_fn, rounds_total)
        e7.record(stream)
        torch.cuda.synchronize()
        stream_total = {"rounds": rounds_total, "seconds": e6.elapsed_time(e7) * 1e-3,
                        "note": "1000 consecutive hs_round steps (HIP graph replays, learner "
                                "state carried), inputs rotating over %d resident rounds; "
                                "generation and host-to-device copies excluded" % copies}

    # ---- the evaluation kernel alone (hs_eval_alpha), live, on the same stream -------------
    run(eval_fn, copies)
    torch.cuda.synchronize()
    e2 = torch.cuda.Event(enable_timing=True)
    e3 = torch.cuda.Event(enable_timing=True)
    e2.record(stream)
    run(eval_fn, n_eval)
    e3.record(stream)
    torch.cuda.synchronize()
    eval_us = e2.elapsed_time(e3) * 1e3 / n_eval
    achieved = w.input_bytes / (eval_us * 1e-6) / 1e9

    if args.copy_calibration:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    read_cal = None
    if args.read_calibration:
        # hs_stream_read over the resident inputs (every byte read once, one word per wave
        # written): the best of a few launch shapes is this device's streaming read rate
        outw = torch.empty(8192 * 4, dtype=torch.int32, device=dev)
        flat = [b.view(-1) for b in bufs]
        shapes = [(g, u, nt) for g in (1024, 2048, 4096, 8192) for u in (2, 4, 8) for nt in (0, 1)]
        best = None
        for g, u, nt in shapes:
            with torch.cuda.stream(stream):
                for t in flat:
                    hs.stream_read(t, grid=g, unroll=u, nontemporal=bool(nt), out=outw,
                                   stream=stream)
            torch.cuda.synchronize()
            e4 = torch.cuda.Event(enable_timing=True)
            e5 = torch.cuda.Event(enable_timing=True)
            reps = 3
            with torch.cuda.stream(stream):
                e4.record(stream)
                for _ in range(reps):
                    for t in flat:
                        hs.stream_read(t, grid=g, unroll=u, nontemporal=bool(nt), out=outw,
                                       stream=stream)
                e5.record(stream)
            torch.cuda.synchronize()
            us = e4.elapsed_time(e5) * 1e3 / (reps * copies)
            if best is None or us < best[0]:
                best = (us, g, u, nt)
        rd_us, g, u, nt = best
        read_cal = {"GBps": w.input_bytes / (rd_us * 1e-6) / 1e9, "us_per_pass": rd_us,
                    "frac_of_peak": w.input_bytes / (rd_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                    "kernel": "hs_stream_read over the %d-byte input of one step, best of %d "
                              "launch shapes: grid %d, %d loads in flight per thread%s"
                              % (w.input_bytes, len(shapes), g, u, ", nontemporal" if nt else "")}

    cpu = cpu_baseline(args, w, np, synth, greedy) if args.cpu_seconds > 0 else None

    name = w.name if args.stack == 1 else "%s_x%d" % (w.name, args.stack)
    line = {
        "metric": METRIC, "value": value, "unit": "drafter-positions/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "N": w.N, "K": w.K, "V": w.V,
                   "logits": logit_type(w),
                   "temperature": w.temperature, "mode": "greedy" if greedy else "sample",
                   "loss": ("length", "accept_token", "accept_chunk")[w.loss],
                   "learners": "hedge+normalhedge", "tree": bool(w.tree),
                   "stacked_instances": args.stack, "rotation_copies": copies,
                   "input_bytes_per_step": w.input_bytes, "hip_graph": use_graph,
                   "wall_s": round(wall, 4)},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic(profile_name(w, name)),
                     "kernel": "hs_eval_alpha = hs_team_kernel (one launch)",
                     "kernel_us": eval_us, "kernel_calls_timed": n_eval,
                     "algorithmic_bytes_per_launch": w.input_bytes,
                     "step_us": ms_step * 1e3},
        "cpu_baseline": cpu,
    }
    if read_cal is not None:
        line["read_calibration"] = read_cal
    if stream_total is not None:
        line["stream_total"] = stream_total
    print(json.dumps(line), flush=True)


def cpu_baseline(args, w, np, synth, greedy):
    """The float64 oracle (alpha or agreement, EAL, loss, Hedge, NormalHedge) on the host, on a
    bounded sample of the same workload: whole queries of round 0 (all N drafters and K
    positions each), first on every core for two thirds of the budget, then on one thread."""
    import oracle

    nq = min(w.B, 4)
    x = synth.generate(synth.variant(w, B=nq), round=0)  # the first nq queries of round 0
    units = [np.ascontiguousarray(x[:, b:b + 1]) for b in range(nq)]
    del x
    par = w.parent()
    pe = w.path_end()

    def one(i):
        b = i % nq
        ref = oracle.evaluate(units[b], V=w.V, T=w.temperature, want_alpha=not greedy)
        gam = (ref["agree"].astype(np.float64) if greedy else ref["alpha"]).transpose(0, 2, 1)
        acc = oracle.accept_len(gam, parent=par, path_end=None if pe is None else pe[b:b + 1],
                                loss_kind=w.loss)
        wo = oracle.hedge(np.full((1, w.N), 1.0 / w.N), acc["loss"], w.eta)
        oracle.normalhedge(np.zeros((1, w.N)), np.full((1, w.N), 1.0 / w.N), acc["loss"])
        return wo

    def timed(budget, min_units=1):
        t1 = time.perf_counter()
        n = 0
        while True:
            one(n)
            n += 1
            el = time.perf_counter() - t1
            if el >= budget and n >= min_units:
                return n, el

    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    threads = min(threads, os.cpu_count() or threads)
    oracle.set_threads(threads)
    n_all, el_all = timed(args.cpu_seconds * 2.0 / 3.0)
    oracle.set_threads(1)
    n_one, el_one = timed(args.cpu_seconds / 3.0)
    oracle.set_threads(threads)
    per_unit = w.N * w.K
    unit_bytes = w.R * w.K * w.V * w.elem_bytes
    return {"value": per_unit * n_all / el_all, "unit": "drafter-positions/s", "cores": threads,
            "kind": "oracle",
            "input_GBps": unit_bytes * n_all / el_all / 1e9,
            "single_thread": {"value": per_unit * n_one / el_one, "unit": "drafter-positions/s",
                              "cores": 1, "input_GBps": unit_bytes * n_one / el_one / 1e9,
                              "queries": n_one, "seconds": round(el_one, 2)},
            "sample": "%d evaluations of whole queries (all %d drafters x %d positions each, "
                      "%.1f MB of logits each), cycling over the first %d queries of round 0 of "
                      "the same workload: float64 C oracle (softmax statistics, alpha or "
                      "agreement, EAL, loss, Hedge, NormalHedge), OpenMP over rows on %d "
                      "threads, %.1f s; then %d on 1 thread, %.1f s"
                      % (n_all, w.N, w.K, unit_bytes / 1e6, nq, threads, el_all, n_one, el_one)}


if __name__ == "__main__":
    main()
