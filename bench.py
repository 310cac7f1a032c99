#!/usr/bin/env python3
"""Throughput of the Hotline hot path on one MI355X.

A step is one pass of the whole per-mini-batch path over one batch: global ids,
classification, partition into popular / non-popular mu-batches, remap, cold
gather for the non-popular mu-batch, forward of both mu-batches and one
coalesced SGD step, in the paper's pipelined schedule: the host-link fetch on
compute units of its own, the next mini-batch's segregation (dispatch, cold
plan, grouping) during the step before on others, the forwards and the
backward on the rest.  The learning phase (access counting over 16 profiling
batches, top-K selection, hot-cache fill) runs once before and is reported
separately.  Inputs (32 measured batches, their gradients, the host table) are
resident before the timed region starts.

Regions, in order: a statistics pass, warmup, the timed region (K steps, no
events inside), then the same steps with HIP events around the kernels of one
name at a time (per-kernel durations for the roofline and the fwd+bwd
fraction), and the oracle's CPU baseline.  --breakdown adds reference
schedules and a per-stage breakdown.

Prints one JSON line on stdout; progress goes to stderr."""
import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "embedding lookups/sec (fwd+bwd) + classify samples/sec; % of HBM peak GB/s"
HBM_PEAK = 8.0e12          # MI355X HBM3E, bytes/s
LINK_PEAK = 64.0e9         # PCIe Gen5 x16, one direction, bytes/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_bytes(name, st, alone=False):
    """Algorithmic bytes of one launch of kernel `name` (per-step statistics
    st): each input read once, each output written once.  L lookups, nb bags,
    B samples, U distinct rows, C distinct cold rows, Lc cold lookups, R bytes
    per stored row, O bytes per pooled output row.  alone: the kernels of the
    calls in order on one stream (the forward over every bag, the whole
    backward: every distinct row read and written by the reduction), else
    those of the pipelined step (hot and cold halves apart)."""
    L, nb, B, U, R, O = st["L"], st["n_bags"], st["B"], st["U"], st["R"], st["O"]
    C, Lc = st["n_cold"], st["Lc"]
    if alone:
        return {
            # the forward over every bag: codes, offsets, each referenced row once, outputs
            "eb_fwd": 4 * L + 4 * (nb + 1) + U * R + nb * O,
            # grouping by table: codes and offsets in, table-major keys out;
            # the keys in, the (key, bag) pairs out
            "gt_prep": 4 * L + 4 * (nb + 1) + 4 * L,
            "gt_sort": 12 * L,
            # the forward and the tables' sorts in one launch
            "eb_fwd_gt": 4 * L + 4 * (nb + 1) + U * R + nb * O + 12 * L,
            "bw_prep_hist": 4 * L + 4 * (nb + 1) + 8 * L,
            "srt_hist": 4 * L,
            "srt_pass": 16 * L,
            # reduction: sorted keys and bags, dY, each updated row read and written
            "bw_reduce1": 8 * L + nb * O + 2 * U * R,
        }.get(name)
    return {
        # rows, offsets, a bitmap word per lookup; gids, codes, flags, the two lists
        "ds_kernel": 4 * L + 4 * (nb + 1) + 8 * L + 8 * L + 5 * B,
        # cold plan: gids and codes of every lookup, table slot per cold lookup, the cold list
        "cg_insert": 8 * L + 8 * Lc,
        "cg_rank": 8 * L + 4 * C,
        "cg_codes": 8 * Lc + 4 * C,
        # the host-link copy (also reported against the link's peak)
        "cg_fetch": 4 * C + 2 * C * R,
        # grouping: keys and bags out (with the fused plan's cold codes: a slot
        # read and a code written per cold lookup), a histogram read, the
        # pairs in and out per pass
        "bw_prep": 4 * L + 4 * (nb + 1) + 8 * L,
        "srt_hist": 4 * L,
        "bw_prep_hist": 4 * L + 4 * (nb + 1) + 8 * L + 8 * Lc,
        "srt_pass": 16 * L,
        "gt_prep": 4 * L + 4 * (nb + 1) + 4 * L + 8 * Lc,
        "gt_sort": 12 * L,
        # hot half of the forward over every bag: codes, offsets, each referenced row once, outputs
        "eb_fwd_hot": 4 * L + 4 * (nb + 1) + (U - C) * R + nb * O,
        # cold half: tail keys and bags, offsets, staging rows, outputs read and written
        "eb_fwd_tail": 8 * Lc + 8 * Lc + C * R + 2 * Lc * O,
        # the same with the reduction's spanning segments (their partial sums are
        # workspace, not algorithmic bytes)
        "eb_tail_r2": 8 * Lc + 8 * Lc + C * R + 2 * Lc * O,
        # the cold half bag by bag (multi-hot): codes and offsets of every bag,
        # staging rows, outputs read and written
        "eb_bags_r2": 4 * L + 4 * (nb + 1) + C * R + 2 * nb * O,
        # reduction: sorted keys and bags, dY, each updated hot row read and
        # written, the staging rows' sums written
        "bw_reduce1": 8 * L + nb * O + 2 * (U - C) * R + C * O,
        "bw_cold": 4 * Lc + 2 * C * R + C * O,
    }.get(name)


def reference_regions(hp, dmeas, side, K):
    """--breakdown: steps tied to the issuing stream, untied steps without
    look-ahead, the fwd+bwd section of the Python rendering (events after the
    fetch and after the backward), and the calls in order on one stream with
    events between the stages."""
    import torch
    from paper_2204_05436_amd.runner import STAGES
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out = {}
    with torch.cuda.stream(side):
        e0.record()
        for i in range(K):
            hp.step(dmeas[i % len(dmeas)])
        e1.record()
    torch.cuda.synchronize()
    out["tied_ms_per_step"] = e0.elapsed_time(e1) / K
    with torch.cuda.stream(side):
        e0.record()
        for i in range(K):
            hp.step(dmeas[i % len(dmeas)], untied=True)
        hp.sync()
        e1.record()
    torch.cuda.synchronize()
    out["untied_no_lookahead_ms_per_step"] = e0.elapsed_time(e1) / K
    evf = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K)]
    for i in range(K):
        hp.step(dmeas[i % len(dmeas)], events=evf[i], mode="fwdbwd")
    torch.cuda.synchronize()
    fb = [e[0].elapsed_time(e[1]) for e in evf]
    out["fwd_bwd_section_us_mean"], out["fwd_bwd_section_us_median"] = 1e3 * np.mean(fb), 1e3 * np.median(fb)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(STAGES) + 1)] for _ in range(K)]
    for i in range(K):
        hp.step(dmeas[i % len(dmeas)], events=ev[i], mode="sequential", split_fwd=False)
    torch.cuda.synchronize()
    st = {s: 0.0 for s in STAGES}
    for i in range(K):
        for j, s in enumerate(STAGES):
            st[s] += ev[i][j].elapsed_time(ev[i][j + 1])
    out["sequential_stages_ms"] = {s: v / K for s, v in st.items()}
    log(f"[bench] breakdown: {out}")
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="dlrm-large")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--repeats", type=int, default=20, help="more timed regions, for the spread of the step time")
    ap.add_argument("--breakdown", action="store_true", help="also time reference schedules and the stages")
    ap.add_argument("--no-relearn", action="store_true", help="skip the timed re-learning (hot-set migration)")
    ap.add_argument("--fetch-study", action="store_true",
                    help="sweep the hot-set size: popular share, cold rows, step time with and without write-back, "
                         "and the share of the host-link fetch hidden under the forward and backward kernels")
    ap.add_argument("--handover-kernels", action="store_true",
                    help="time the steps with the handovers between streams as kernels of their own instead of "
                         "inside the path's kernels (whose first block signals at the start and waits at the end)")
    ap.add_argument("--eal-study", action="store_true", help="compare the SRRIP logger with exact top-K on every workload")
    ap.add_argument("--pmc", action="store_true",
                    help="for a counter run under rocprofv3 --pmc: warmup + --steps steps of the same kernels on one "
                         "stream, then one device copy of known size (the counters' calibration); prints that size "
                         "and exits")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the path shards "
              "by samples across GPUs but no multi-GPU run is part of it", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2204_05436_amd import configs, hotline as hl, workload as W
    from paper_2204_05436_amd.runner import HotPath, to_device

    dev = "cuda:0"
    torch.cuda.set_device(0)
    w = configs.WORKLOADS[args.workload]
    rows = W.table_rows(w)
    n_rows = int(rows.sum(dtype=np.int64))
    k_cap = w.k_cap(n_rows)
    log(f"[bench] workload {w.name}: {w.n_tables} tables, {n_rows} rows, dim {w.dim} {w.dtype}, batch {w.batch}")
    t0 = time.time()
    prof = [W.make_batch(w, rows, i) for i in range(w.profile_batches)]
    meas_idx = list(range(w.profile_batches, w.profile_batches + w.measured_batches))
    meas = [W.make_batch(w, rows, i) for i in meas_idx]
    log(f"[bench] batches generated in {time.time() - t0:.1f}s")
    table = hl.HostTable(n_rows, w.dim, w.dtype)
    t0 = time.time()
    W.fill_weights_torch(w, table.torch_view(), dev)
    torch.cuda.synchronize()
    log(f"[bench] host table {table.nbytes / 2**30:.2f} GiB pinned+filled in {time.time() - t0:.1f}s")
    dprof = [to_device(b, dev) for b in prof]
    dmeas = []
    for i, b in zip(meas_idx, meas):
        dmeas.append(to_device(b, dev, W.make_dy(w, i, b.n_bags)))
    max_l = max(b.n_lookups for b in prof + meas)
    # (the study's smaller hot sets leave up to every row of a mini-batch cold)
    # (a counter run serializes dispatches, so its path takes no masked streams:
    # their flag handovers, and the pipeline's check of them, would stall)
    hp = HotPath(w, rows, table, max_l, w.batch, device=dev, staging_cap=max_l if args.fetch_study else None,
                 fetch_cus=0 if args.pmc else 8)
    log(f"[bench] inputs resident; workspace {hp.ws.numel() / 2**20:.1f} MiB, hot cache {k_cap} rows")

    # learning phase
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    n_hot = hp.learn(dprof)
    e1.record()
    torch.cuda.synchronize()
    learn_ms = e0.elapsed_time(e1)
    log(f"[bench] learning phase {learn_ms:.2f} ms, n_hot {n_hot}")

    if args.pmc:
        # the step's kernels one at a time on one stream (a counter run
        # serializes dispatches, which the pipelined schedule's cross-stream
        # waits would stall on), through the calls that launch the same kernel
        # variants as the pipelined step where the library has them: the hot
        # half of the forward over every sample, the grouping, the split
        # reduction, the staging-row updates and the host-link copy; then the
        # forward and backward of the calls in order
        h = hp.h
        for i in range(args.warmup + args.steps):
            b = dmeas[i % len(dmeas)]
            B, bps, L, cap = b.n_samples, b.bps, b.n_lookups, hp.staging_cap
            hl.hl_dispatch(h, b.rows, b.bag_ptr, B, bps, L, hp.gids, hp.codes, hp.flags, hp.pop, hp.nonpop,
                           hp.counts, hp.ws)
            hl.hl_cold_plan(h, hp.gids, hp.codes, b.bag_ptr, B, bps, L, None, None, B, cap, hp.cold_ids, hp.n_cold,
                            hp.ws)
            hl.hl_cold_fetch(h, hp.cold_ids, hp.n_cold, cap, table.dev, hp.staging)
            hl.hl_embbag_bwd_plan(h, cap, hp.codes, b.bag_ptr, B, bps, L, None, None, B, hp.ws)
            hl.hl_embbag_fwd_part(h, hp.w_hot, hp.staging, cap, hp.codes, b.bag_ptr, B, bps, L, None, None, B,
                                  hp.out, 1)
            hl.hl_embbag_bwd_apply_part(h, hp.w_hot, hp.staging, cap, B, bps, L, b.dY, w.lr, 1, hp.ws)
            hl.hl_embbag_fwd_part(h, hp.w_hot, hp.staging, cap, hp.codes, b.bag_ptr, B, bps, L, hp.nonpop,
                                  hp.counts[1:], B, hp.out, 2)
            hl.hl_embbag_bwd_apply_part(h, hp.w_hot, hp.staging, cap, B, bps, L, b.dY, w.lr, 2, hp.ws)
            # the variants of the calls in order on one stream: the forward over
            # every bag with the backward's plan, then the apply
            hl.hl_embbag_fwd_plan(h, hp.w_hot, hp.staging, cap, hp.codes, b.bag_ptr, B, bps, L, hp.out, hp.ws)
            hl.hl_embbag_bwd_apply(h, hp.w_hot, hp.staging, cap, B, bps, L, b.dY, w.lr, hp.ws)
        torch.cuda.synchronize()
        n_cal = 256 << 20
        src = torch.ones(n_cal // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        err = hp.device_error()
        print(json.dumps({"mode": "pmc", "workload": w.name, "steps": args.warmup + args.steps, "device_error": err,
                          "calibration_copy_bytes": n_cal}), flush=True)
        hp.close()
        table.close()
        return

    # per-batch statistics (untimed pass over every measured batch)
    # steps are issued from a stream of their own (work on the default stream
    # would serialize with the pipeline's streams)
    side = torch.cuda.Stream()

    def ahead(i, n):
        """the batches after step i of n that the runner plans ahead"""
        return [dmeas[(i + j) % len(dmeas)] for j in range(1, hp.n_sets) if i + j < n]
    stats = []
    for j, b in enumerate(dmeas):
        with torch.cuda.stream(side):
            hp.step(b, next=ahead(j, len(dmeas)))
        torch.cuda.synchronize()
        L = b.n_lookups
        U = int(torch.unique(hp.codes[:L]).numel())
        c = hp.counts.cpu().numpy()
        Lc = int((hp.codes[:L] >= hp.k_cap).sum().item())
        stats.append(dict(L=L, n_bags=b.n_bags, B=b.n_samples, U=U, n_pop=int(c[0]), n_cold=int(hp.n_cold.item()),
                          Lc=Lc, R=hp.staging.element_size() * w.dim, O=4 * w.dim))
    err = hp.device_error()
    if err:
        raise SystemExit(f"device error word {err:#x} after the statistics pass")
    log("[bench] statistics pass done")
    hk = args.handover_kernels
    with torch.cuda.stream(side):
        for i in range(args.warmup):
            hp.step(dmeas[i % len(dmeas)], untied=True, next=ahead(i, args.warmup), handover_kernels=hk)
        hp.sync()
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup} steps done")
    K = args.steps

    # timed region: K pipelined steps back to back (inputs resident, so the steps
    # are not tied to the issuing stream; one wait for all of them at the end),
    # nothing but the path (no events inside).  Each step plans the next batch
    # (its dispatch and cold plan run while the step trains), so the region
    # holds K plans (batches 0..K-1) and K steps.
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(side):
        t_start = time.perf_counter()
        start.record()  # the side stream is idle: the event completes before the first step is issued
        for i in range(K):
            hp.step(dmeas[i % len(dmeas)], untied=True, next=ahead(i, K), handover_kernels=hk)
        host_ms = (time.perf_counter() - t_start) * 1e3
        hp.sync()
        stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    total_ms = start.elapsed_time(stop)
    log(f"[bench] timed {K} steps: {total_ms:.3f} ms (wall {wall * 1e3:.1f} ms, host enqueue {host_ms:.1f} ms)")
    err = hp.device_error()
    if err:
        raise SystemExit(f"device error word {err:#x} in the timed region")

    # the same region repeated
    reps = []
    for r in range(args.repeats):
        with torch.cuda.stream(side):
            start.record()
            for i in range(K):
                hp.step(dmeas[i % len(dmeas)], untied=True, next=ahead(i, K), handover_kernels=hk)
            hp.sync()
            stop.record()
        torch.cuda.synchronize()
        reps.append(start.elapsed_time(stop) / K)
    err = hp.device_error()
    if err:
        raise SystemExit(f"device error word {err:#x} in the repeated regions")
    # the line's time per step: the median over all regions (the first one
    # included), with p10/p90 beside it
    first_ms = total_ms / K
    reps = [first_ms] + reps
    spread = {"regions": len(reps), "median": float(np.median(reps)), "p10": float(np.percentile(reps, 10)),
              "p90": float(np.percentile(reps, 90)), "first_region": first_ms}
    total_ms = spread["median"] * K
    log(f"[bench] {len(reps)} regions of {K} steps: ms per step median {spread['median']:.4f} "
        f"(p10 {spread['p10']:.4f}, p90 {spread['p90']:.4f}, first region {first_ms:.4f})")

    # achievable HBM rate: a 256 MiB device-to-device copy
    src = torch.empty(64 << 20, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    copy_GBps = 10 * 2 * src.numel() * 4 / (e0.elapsed_time(e1) / 1e3) / 1e9
    del src, dst
    # achievable host-link rate: a pinned host buffer copied to the device, of
    # the cold rows' size per step and of 64 MiB
    h2d_GBps = {}
    for nbytes in (max(4096, int(np.mean([s["n_cold"] * s["R"] for s in stats]))), 64 << 20):
        hsrc = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
        ddst = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        ddst.copy_(hsrc, non_blocking=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(10):
            ddst.copy_(hsrc, non_blocking=True)
        e1.record()
        torch.cuda.synchronize()
        h2d_GBps[str(nbytes)] = 10 * nbytes / (e0.elapsed_time(e1) / 1e3) / 1e9
        del hsrc, ddst
    log(f"[bench] pinned host-to-device copies: " + ", ".join(f"{k} B {v:.1f} GB/s" for k, v in h2d_GBps.items()))

    steps_stats = [stats[i % len(stats)] for i in range(K)]
    avg = {k: float(np.mean([s[k] for s in steps_stats])) for k in steps_stats[0]}
    L_tot = sum(s["L"] for s in steps_stats)
    value = L_tot / (total_ms / 1e3)

    def look_ahead_steps(hk):
        with torch.cuda.stream(side):
            for i in range(K):
                hp.step(dmeas[i % len(dmeas)], untied=True, next=ahead(i, K), handover_kernels=hk)
            hp.sync()
        torch.cuda.synchronize()

    def sequential_steps():
        with torch.cuda.stream(side):
            for i in range(K):
                hp.step(dmeas[i % len(dmeas)], mode="sequential", split_fwd=False)
        torch.cuda.synchronize()

    def traced(run, only):
        """K steps of `run` with every kernel named `only` (None: every kernel)
        timed by its own dispatch (events that the launch itself records);
        per name: launches and total ms."""
        hl.hl_trace_enable(hp.h, 64 * K + 64)
        hl.hl_trace_only(hp.h, only)
        run()
        kern = {}
        for i in range(hl.hl_trace_count(hp.h)):
            name, ms = hl.hl_trace_read(hp.h, i)
            k = kern.setdefault(name, [0, 0.0])
            k[0] += 1
            k[1] += ms
        hl.hl_trace_only(hp.h, None)
        hl.hl_trace_enable(hp.h, 0)
        err = hp.device_error()
        if err:
            raise SystemExit(f"device error word {err:#x} in a traced pass")
        return kern

    def per_kernel(run, alone):
        """which kernels run (all traced), then each name traced alone"""
        kern = {}
        for n in traced(run, None):
            c, t = traced(run, n)[n]
            kern[n] = {"launches_per_step": c / K, "ms_per_step": t / K, "avg_us": 1e3 * t / c}
            kb = kernel_bytes(n, avg, alone)
            if kb is not None:
                kern[n]["algorithmic_GBps"] = kb / (kern[n]["avg_us"] * 1e-6) / 1e9
        return dict(sorted(kern.items(), key=lambda x: -x[1]["ms_per_step"]))

    def fmt(kern):
        return ", ".join(f"{n} {k['avg_us']:.1f}us x{k['launches_per_step']:.0f}" for n, k in kern.items())

    # per-kernel durations: in the timed schedule (with the handovers inside
    # the kernels, a kernel's duration includes its waits for the other
    # streams), in the same schedule with the handovers as kernels of their
    # own (each kernel's own work, beside the other streams' kernels), and in
    # the calls in order on one stream (each kernel alone on the whole GPU)
    kernels_timed = per_kernel(lambda: look_ahead_steps(hk), False)
    log("[bench] per-kernel times, timed schedule: " + fmt(kernels_timed))
    kernels = kernels_timed if hk else per_kernel(lambda: look_ahead_steps(True), False)
    if not hk:
        log("[bench] per-kernel times, handovers as kernels: " + fmt(kernels))
    kernels_alone = per_kernel(sequential_steps, True)
    log("[bench] per-kernel times, alone: " + fmt(kernels_alone))

    # the embedding forward and backward: their kernels' time per step (the
    # grouping included), against the algorithmic bytes of both passes
    fb_kernels = ("eb_fwd", "eb_fwd_gt", "eb_fwd_hot", "eb_fwd_tail", "eb_tail_r2", "eb_bags_r2", "bw_prep", "bw_prep_hist",
                  "srt_hist", "srt_pass", "gt_prep", "gt_sort", "bw_reduce1", "bw_reduce2", "bw_cold")
    t_fb = sum(kernels[n]["ms_per_step"] for n in fb_kernels if n in kernels)
    t_fb_alone = sum(kernels_alone[n]["ms_per_step"] for n in fb_kernels if n in kernels_alone)
    fwd_b = 4 * avg["L"] + 4 * (avg["n_bags"] + 1) + avg["U"] * avg["R"] + avg["n_bags"] * avg["O"]
    bwd_b = 4 * avg["L"] + 4 * (avg["n_bags"] + 1) + avg["n_bags"] * avg["O"] + 2 * avg["U"] * avg["R"]
    fb_frac = (fwd_b + bwd_b) / (t_fb / 1e3) / HBM_PEAK
    fb_frac_alone = (fwd_b + bwd_b) / (t_fb_alone / 1e3) / HBM_PEAK

    # roofline of the dominant HBM-bound kernel of the forward and backward,
    # by time per step alone on the GPU (its own work, no wait for another
    # stream inside it; rocprofv3 sees these launches under their own kernel
    # names, apart from the pipelined step's variants): the forward and the
    # backward's reduction move the path's bytes; the grouping is
    # latency-bound at these sizes.  Then the same for the timed schedule's
    # dominant HBM-bound kernel, from the pass with its handovers as kernels
    # of their own (beside the other streams' kernels, on the main stream's
    # compute units), and the dominant kernel overall.
    def roofline(kern, names, alone):
        dom = next(n for n in kern if n in names)
        kd = kern[dom]
        ab = kernel_bytes(dom, avg, alone)
        if ab is None:
            raise SystemExit(f"no byte model for the dominant kernel {dom}")
        ach = ab / (kd["avg_us"] * 1e-6)
        # measured HBM bytes per launch (counters, same kernel source), as a
        # rate over the same launch duration as `achieved`
        tb = counter_traffic(dom, w.name, alone)
        return {"kernel": dom, "bound": "hbm", "achieved": ach / 1e9, "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                "frac": ach / HBM_PEAK, "traffic": None if tb is None else tb / (kd["avg_us"] * 1e-6) / 1e9,
                "traffic_bytes_per_launch": tb, "avg_us": kd["avg_us"], "algorithmic_bytes_per_launch": ab,
                "schedule": "alone" if alone else "timed, handovers as kernels"}
    roof = roofline(kernels_alone, ("eb_fwd", "eb_fwd_gt", "bw_reduce1", "bw_reduce2"), True)
    roof_timed = roofline(kernels, ("eb_fwd_hot", "bw_reduce1", "bw_reduce2"), False)
    dom_all = next(n for n in kernels if n not in ("cg_fetch", "cg_scatter"))
    roof_timed["dominant_kernel_overall"] = {"kernel": dom_all, "ms_per_step": kernels[dom_all]["ms_per_step"]}
    link = None
    if "cg_fetch" in kernels:
        gb = avg["n_cold"] * avg["R"]
        link = {"kernel": "cg_fetch", "bytes_per_launch": gb, "avg_us": kernels["cg_fetch"]["avg_us"],
                "achieved_GBps": gb / (kernels["cg_fetch"]["avg_us"] * 1e-6) / 1e9, "peak_GBps": LINK_PEAK / 1e9,
                "measured_pinned_copy_GBps": h2d_GBps}

    # the same batches through the library's calls in order on one stream: the
    # spans of classify+partition and of fwd+bwd between events (launch gaps
    # included), then one pass with events between every stage.  Events only
    # at the edges of the spans timed (a pair of events adds a few
    # microseconds of its own: the stages' pass below has an empty span).
    from paper_2204_05436_amd.runner import STAGES
    ix = {s: j for j, s in enumerate(STAGES)}
    edges = (ix["classify"], ix["remap"], ix["fwd_pop"], len(STAGES))  # classify+partition, fwd+bwd

    class _NoEvent:
        def record(self, *a):
            pass

    def seq_pass(marks):
        ev = [[torch.cuda.Event(enable_timing=True) if j in marks else _NoEvent() for j in range(len(STAGES) + 1)]
              for _ in range(K)]
        with torch.cuda.stream(side):
            for i in range(K):
                hp.step(dmeas[i % len(dmeas)], events=ev[i], mode="sequential", split_fwd=False)
        torch.cuda.synchronize()
        err = hp.device_error()
        if err:
            raise SystemExit(f"device error word {err:#x} in the sequential steps")
        return ev

    ev = seq_pass(edges)
    t_cp = sum(e[edges[0]].elapsed_time(e[edges[1]]) for e in ev) / K
    t_fb1 = sum(e[edges[2]].elapsed_time(e[edges[3]]) for e in ev) / K
    ev = seq_pass(range(len(STAGES) + 1))
    st = {s: sum(ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(K)) / K for j, s in enumerate(STAGES)}
    cl_kern = ("hl_k_gids", "cl_kernel", "pt_count", "pt_scan", "pt_emit", "pt_one")
    t_cl_alone = sum(kernels_alone[n]["ms_per_step"] for n in cl_kern if n in kernels_alone)
    alone = {"fwd_bwd_kernel_us": t_fb_alone * 1e3, "fwd_bwd_lookups_per_s": avg["L"] / (t_fb_alone / 1e3),
             "fwd_bwd_hbm_frac": fb_frac_alone,
             "fwd_bwd_span_us": t_fb1 * 1e3, "fwd_bwd_span_hbm_frac": (fwd_b + bwd_b) / (t_fb1 / 1e3) / HBM_PEAK,
             # every lookup's row counted (no coalescing): fwd L R + n O, bwd n O + 2 L R
             "lookup_equivalent_GBps": (3 * avg["L"] * avg["R"] + 2 * avg["n_bags"] * avg["O"]) / (t_fb_alone / 1e3)
             / 1e9,
             "achievable_copy_GBps": copy_GBps,
             "classify_partition_kernel_us": t_cl_alone * 1e3,
             "classify_samples_per_s": avg["B"] / (t_cl_alone / 1e3) if t_cl_alone else None,
             "classify_partition_span_us": t_cp * 1e3,
             "stage_ms_events_between_every_stage": st,
             "empty_span_us": st["fwd_nonpop"] * 1e3,
             "kernels": kernels_alone}
    log(f"[bench] alone on the GPU: fwd+bwd kernels {t_fb_alone * 1e3:.1f} us ({fb_frac_alone:.3f} of the HBM "
        f"peak; span {t_fb1 * 1e3:.1f} us), classify+partition kernels {t_cl_alone * 1e3:.1f} us; stages " +
        ", ".join(f"{s} {v * 1e3:.1f}us" for s, v in st.items()))

    breakdown = None
    if args.breakdown:
        breakdown = reference_regions(hp, dmeas, side, K)

    # the learning phase again (after the measured steps, so it changes nothing
    # above): counts over a sample of batches whose popularity has drifted (the
    # same Zipf ranks on other rows), the new top-K, and the hot-cache migration
    # the SRRIP access logger against the exact hot set learnt above, at its size
    eal = eal_compare(hp.h, dprof, dmeas[:8], hp.hot_ids[:hp.n_hot].clone(), hp.n_hot)
    log(f"[bench] SRRIP logger ({eal['sets']} sets x {eal['ways']} ways): holds {eal['captured_frac']:.3f} of the "
        f"exact hot set; lookups hot {eal['lookups_hot_frac']['srrip']:.3f} vs {eal['lookups_hot_frac']['exact']:.3f}; "
        f"{eal['us_per_batch']:.1f} us per batch")
    eal_all = None
    if args.eal_study:
        eal_all = {}
        eal_study(eal_all)

    # the timed region again with the write-back of the updated cold rows to
    # the host table (on the fetch stream after each step; the next plans and
    # fetches of those rows wait for it)
    def timed_steps(n):
        with torch.cuda.stream(side):
            start.record()
            for i in range(n):
                hp.step(dmeas[i % len(dmeas)], untied=True, next=ahead(i, n), handover_kernels=hk)
            hp.sync()
            stop.record()
        torch.cuda.synchronize()
        err = hp.device_error()
        if err:
            raise SystemExit(f"device error word {err:#x} in a timed region")
        return start.elapsed_time(stop) / n

    hp.writeback = True
    timed_steps(args.warmup)
    wb_ms = float(np.median([timed_steps(K) for _ in range(5)]))
    wb_kern = traced(lambda: look_ahead_steps(hk), "cg_scatter").get("cg_scatter", [0, 0.0])
    hp.writeback = False
    write_back = {"ms_per_step": wb_ms, "lookups_per_s": L_tot / K / (wb_ms / 1e3),
                  "cg_scatter_avg_us": 1e3 * wb_kern[1] / max(1, wb_kern[0]),
                  "bytes_per_step": avg["n_cold"] * avg["R"]}
    log(f"[bench] with write-back: {wb_ms:.4f} ms per step (without {total_ms / K:.4f}), write-back copy "
        f"{write_back['cg_scatter_avg_us']:.1f} us")

    study = fetch_study(hp, w, dprof, dmeas, side, K, ahead, traced, look_ahead_steps) if args.fetch_study else None

    relearn = None
    if not args.no_relearn:
        drift = [to_device(W.make_batch(w, rows, 1000 + i, phase=1), dev) for i in range(w.profile_batches)]
        old = hp.hot_ids[:hp.n_hot].cpu().numpy()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        n_new = hp.relearn(drift)
        torch.cuda.synchronize()
        rl_ms = (time.perf_counter() - t0) * 1e3
        new = hp.hot_ids[:n_new].cpu().numpy()
        err = hp.device_error()
        if err:
            raise SystemExit(f"device error word {err:#x} in the re-learning")
        leave, enter = int(np.setdiff1d(old, new).size), int(np.setdiff1d(new, old).size)
        relearn = {"ms": rl_ms, "sampled_batches": len(drift), "n_hot_before": int(old.size), "n_hot": int(n_new),
                   "rows_written_back": leave, "rows_entered": enter, "steps_equivalent": rl_ms / (total_ms / K)}
        log(f"[bench] re-learning over {len(drift)} drifted batches: {rl_ms:.2f} ms, {leave} rows left the cache, "
            f"{enter} entered")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, rows, prof, meas, meas_idx, table, k_cap, args.cpu_seconds)

    res = {
        "metric": METRIC, "value": value, "unit": "lookups/s", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": total_ms / K, "ms_per_step_spread": spread, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name, "tables": w.n_tables, "rows": n_rows, "dim": w.dim, "storage": w.dtype,
                   "batch": w.batch, "bags_per_sample": w.bags_per_sample, "lookups_per_batch": avg["L"],
                   "zipf_alpha": w.alpha, "hot_cache_rows": k_cap, "n_hot": n_hot,
                   "profile_batches": w.profile_batches, "measured_batches": w.measured_batches,
                   "parallelism": "single-gpu"},
        "schedule": "pipelined by the native scheduler: the host-link fetch on 8 compute units, the look-ahead "
                    "plans (dispatch, cold plan, grouping of the next mini-batch, during the step before) on 64, "
                    "the forwards and the backward on the other 184",
        "host_enqueue_ms_per_step": host_ms / K,
        "handovers": "kernels" if hk else "inline",
        # the forward and backward kernels' own work per step in the timed
        # schedule (handovers as kernels), and against their time alone
        "fwd_bwd_kernel_us": t_fb * 1e3,
        "fwd_bwd_timed_over_alone": t_fb / t_fb_alone,
        "fwd_bwd_lookups_per_s": avg["L"] / (t_fb / 1e3),
        "fwd_bwd_hbm_frac": fb_frac,
        "fwd_bwd_algorithmic_bytes": fwd_b + bwd_b,
        "alone_on_gpu": alone,
        # the dispatch kernel classifies, partitions and remaps a mini-batch
        # the dispatch kernel's own work (classify, partition, remap of a mini-batch)
        "classify_samples_per_s": avg["B"] / (kernels["ds_kernel"]["avg_us"] * 1e-6),
        "classify_kernel_us": kernels["ds_kernel"]["avg_us"],
        "popular_fraction": avg["n_pop"] / avg["B"],
        "unique_rows_per_batch": avg["U"], "cold_rows_per_batch": avg["n_cold"],
        "learning_phase_ms": learn_ms, "kernels": kernels, "kernels_timed_schedule": kernels_timed,
        "roofline": roof, "roofline_timed_schedule": roof_timed, "link_roofline": link, "cpu_baseline": cpu, "breakdown": breakdown, "relearn": relearn,
        "srrip_logger": eal, "srrip_logger_all_workloads": eal_all,
        "write_back": write_back, "fetch_study": study,
    }
    print(json.dumps(res), flush=True)
    hp.close()
    table.close()


# the main stream's kernels of a planned step: the forwards and the backward
MAIN_KERNELS = ("eb_fwd_hot", "eb_fwd_cold", "eb_fwd_tail", "eb_tail_r2", "eb_bags_r2", "bw_reduce1", "bw_reduce2",
                "bw_cold")


def fetch_overlap(hp, run, K):
    """One run with the host-link copy and the main stream's kernels (the
    forwards and the backward) traced, start and end on one time line (the
    other kernels untraced: tracing every kernel changes the schedule): the
    copy's time per launch, the share of it during which a main-stream kernel
    ran, and the run's time per step (to compare with the untraced steps)."""
    import torch
    from paper_2204_05436_amd import hotline as hl
    hl.hl_trace_enable(hp.h, 1 << 16)
    hl.hl_trace_only(hp.h, ",".join(("cg_fetch",) + MAIN_KERNELS))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    run()
    e1.record()
    torch.cuda.synchronize()
    recs = [hl.hl_trace_read_at(hp.h, i) for i in range(hl.hl_trace_count(hp.h))]
    hl.hl_trace_only(hp.h, None)
    hl.hl_trace_enable(hp.h, 0)

    def union(iv):
        out = []
        for a, b in sorted(iv):
            if out and a <= out[-1][1]:
                out[-1][1] = max(out[-1][1], b)
            else:
                out.append([a, b])
        return out

    def covered(f, u):
        return sum(max(0.0, min(f[1], b) - max(f[0], a)) for a, b in u)
    fetch = [(t0, t0 + d) for n, t0, d in recs if n == "cg_fetch"]
    main = union([(t0, t0 + d) for n, t0, d in recs if n in MAIN_KERNELS])
    tf = sum(b - a for a, b in fetch)
    return {"fetch_us": 1e3 * tf / max(1, len(fetch)),
            "hidden_under_fwd_bwd": sum(covered(f, main) for f in fetch) / tf if tf else None,
            "traced_ms_per_step": e0.elapsed_time(e1) / K}


def fetch_study(hp, w, dprof, dmeas, side, K, ahead, traced, look_ahead_steps):
    """Hot sets of 1/32 ... all of the rows the profiling batches touched
    (up to the cache's capacity): per size the popular share of samples, the
    cold rows per mini-batch, the step time without and with write-back, and
    the share of the fetch hidden under the forward and backward kernels
    (Sec. VII-F: the popular share decides how much of the gather the
    pipeline hides)."""
    import torch
    n_full = hp.learn(dprof)
    out = []
    for frac in (1 / 32, 1 / 8, 1 / 4, 1 / 2, 1):
        k = max(1, int(n_full * frac))
        n_hot = hp.learn(dprof, k=k)
        pops, colds = [], []
        for j, b in enumerate(dmeas[:8]):
            with torch.cuda.stream(side):
                hp.step(b)
            torch.cuda.synchronize()
            c = hp.counts.cpu().numpy()
            pops.append(c[0] / b.n_samples)
            colds.append(int(hp.n_cold.item()))
        ms = {}
        for wb in (False, True):
            hp.writeback = wb
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            look_ahead_steps(False)
            with torch.cuda.stream(side):
                e0.record()
                for i in range(K):
                    hp.step(dmeas[i % len(dmeas)], untied=True, next=ahead(i, K))
                hp.sync()
                e1.record()
            torch.cuda.synchronize()
            ms["with_write_back" if wb else "no_write_back"] = e0.elapsed_time(e1) / K
        hp.writeback = False
        ov = fetch_overlap(hp, lambda: look_ahead_steps(False), K)
        err = hp.device_error()
        if err:
            raise SystemExit(f"device error word {err:#x} in the fetch study")
        row = {"hot_rows": n_hot, "popular_share": float(np.mean(pops)), "cold_rows_per_batch": float(np.mean(colds)),
               "ms_per_step": ms, **ov}
        log(f"[bench] fetch study: {row}")
        out.append(row)
    hp.learn(dprof)
    return out


def counter_traffic(kernel, workload, alone=False):
    """HBM bytes per launch of `kernel` (alone: its variant in the calls in
    order on one stream, else the pipelined step's) from the committed
    counter summary (profiles/<workload>_kernel_traffic.md: FETCH_SIZE and
    WRITE_SIZE runs, calibrated with a copy of known size), or None when there
    is none or the kernel's source file has changed since the counters were
    taken."""
    here = os.path.dirname(os.path.abspath(__file__))
    path = os.path.join(here, "profiles", f"{workload}_kernel_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"```traffic_alone\n(.*?)```" if alone else r"```traffic\n(.*?)```", text, re.S)
    if not m:
        return None
    # a line: kernel, bytes per launch, then (source file, sha1) pairs of the
    # files its code comes from
    for line in m.group(1).splitlines():
        f = line.split()
        if len(f) >= 4 and len(f) % 2 == 0 and f[0] == kernel:
            srcs = [(os.path.join(here, f[i]), f[i + 1]) for i in range(2, len(f), 2)]
            if all(os.path.exists(p) and hashlib.sha1(open(p, "rb").read()).hexdigest() == h for p, h in srcs):
                return int(f[1])
    return None


def eal_compare(h, prof, meas, exact, capacity, ways=16):
    """The SRRIP access logger (hl_eal_*) against exact counting at the same
    capacity: the logger gets floor(capacity / ways) sets and the profiling
    batches (device batches), and its hot set is compared with the exact one
    (device ids): the share of the exact set it holds, and the share of the
    measured batches' lookups, and of their samples (popular: every lookup hot),
    each set covers.  Also the logger's time per batch (HIP events)."""
    import torch
    from paper_2204_05436_amd import hotline as hl
    n_sets = max(1, capacity // ways)
    max_l = max(b.n_lookups for b in prof + meas)
    e = hl.EAL(h, n_sets, ways, max_l)
    gids = torch.zeros(max_l, dtype=torch.int32, device="cuda")
    try:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ms = 0.0
        for b in prof:
            hl.hl_lookup_gids(h, b.rows, b.bag_ptr, b.n_samples * b.bps, gids)
            e0.record()
            hl.hl_eal_access(e, gids, b.n_lookups)
            e1.record()
            torch.cuda.synchronize()
            ms += e0.elapsed_time(e1)
        held = torch.zeros(n_sets * ways, dtype=torch.int32, device="cuda")
        n = hl.hl_eal_hot(e, held)
        held = held[:n]
        sets = {"srrip": held, "exact": exact}
        cov = {k: [0, 0] for k in sets}
        pop = {k: [0, 0] for k in sets}
        for b in meas:
            L = b.n_lookups
            hl.hl_lookup_gids(h, b.rows, b.bag_ptr, b.n_samples * b.bps, gids)
            ptr = b.bag_ptr.long()
            starts, ends = ptr[0:-1:b.bps][:b.n_samples], ptr[b.bps::b.bps][:b.n_samples]
            for k, ids in sets.items():
                hot = torch.isin(gids[:L], ids)
                cov[k][0] += int(hot.sum())
                cov[k][1] += L
                cs = torch.cat([torch.zeros(1, dtype=torch.long, device="cuda"), torch.cumsum((~hot).long(), 0)])
                pop[k][0] += int(((cs[ends] - cs[starts]) == 0).sum())
                pop[k][1] += b.n_samples
        inter = int(torch.isin(held, exact).sum())
        return {"capacity": n_sets * ways, "sets": n_sets, "ways": ways, "exact_hot": int(exact.numel()),
                "srrip_hot": int(n), "captured_frac": inter / max(1, int(exact.numel())),
                "lookups_hot_frac": {k: v[0] / max(1, v[1]) for k, v in cov.items()},
                "popular_samples_frac": {k: v[0] / max(1, v[1]) for k, v in pop.items()},
                "us_per_batch": ms * 1e3 / max(1, len(prof)),
                "lookups_per_s": sum(b.n_lookups for b in prof) / max(1e-9, ms * 1e-3)}
    finally:
        e.close()


def eal_study(out):
    """The comparison on every workload (full size, 16 profiling batches, 8
    measured ones), capacity = the hot-set size K, 16 ways."""
    import torch
    from paper_2204_05436_amd import configs, hotline as hl, workload as W
    from paper_2204_05436_amd.runner import to_device
    for name in configs.ORDER:
        w = configs.WORKLOADS[name]
        rows = W.table_rows(w)
        n_rows = int(rows.sum(dtype=np.int64))
        k_cap = w.k_cap(n_rows)
        prof = [to_device(W.make_batch(w, rows, i), "cuda") for i in range(w.profile_batches)]
        meas = [to_device(W.make_batch(w, rows, w.profile_batches + i), "cuda") for i in range(8)]
        h = hl.hl_create(rows, w.dim, w.dtype, k_cap)
        try:
            gids = torch.zeros(max(b.n_lookups for b in prof), dtype=torch.int32, device="cuda")
            for b in prof:
                hl.hl_lookup_gids(h, b.rows, b.bag_ptr, b.n_samples * b.bps, gids)
                hl.hl_profile_count(h, gids, b.n_lookups)
            exact = torch.zeros(min(k_cap, n_rows), dtype=torch.int32, device="cuda")
            n_hot = hl.hl_profile_topk(h, k_cap, exact, reset_counts=True)
            r = eal_compare(h, prof, meas, exact[:n_hot], min(k_cap, n_hot))
        finally:
            hl.hl_destroy(h)
        r["k_cap"] = k_cap
        out[name] = r
        log(f"[bench] SRRIP logger on {name}: holds {r['captured_frac']:.3f} of the exact hot set "
            f"({r['exact_hot']} ids, capacity {r['capacity']}); lookups hot {r['lookups_hot_frac']['srrip']:.3f} vs "
            f"{r['lookups_hot_frac']['exact']:.3f}; popular samples {r['popular_samples_frac']['srrip']:.3f} vs "
            f"{r['popular_samples_frac']['exact']:.3f}")


def cpu_baseline(w, rows, prof, meas, meas_idx, table, k_cap, budget_s):
    """The oracle (single-threaded C, fp64) on the same batches, pinned to one
    host core (the calling thread's affinity, restored after): learning phase
    once (untimed), then the per-batch steps timed batch by batch, the measured
    batches over and over, until the budget is spent, with the time of each
    stage beside the total.  The times include the binding's numpy
    marshalling around each oracle call."""
    import oracle as O
    from paper_2204_05436_amd import workload as W

    n_rows = int(rows.sum(dtype=np.int64))
    counts = np.zeros(n_rows, dtype=np.uint32)
    for p in prof:
        g, _ = O.gids(rows, p.rows, p.bag_ptr)
        O.count(n_rows, [g], counts)
    hot = O.topk(counts, k_cap)
    w_hot = O.gather(table.array, hot)
    done, L, B, t_all = 0, 0, 0, 0.0
    stage = {"classify_partition": 0.0, "remap_coldplan_gather": 0.0, "fwd": 0.0, "bwd": 0.0}
    aff = os.sched_getaffinity(0)
    core = min(aff)
    os.sched_setaffinity(0, {core})
    log(f"[bench] cpu baseline (oracle) on core {core} ...")
    try:
        dYs = [W.make_dy(w, i, mb.n_bags) for i, mb in zip(meas_idx, meas)]
        while t_all < budget_s:
            mb, dY = meas[done % len(meas)], dYs[done % len(meas)]
            bps = mb.bags_per_sample
            t0 = time.perf_counter()
            g, _ = O.gids(rows, mb.rows, mb.bag_ptr)
            flags = O.classify(hot, g, mb.bag_ptr, mb.n_samples, bps)
            pop, nonpop = O.partition(flags)
            t1 = time.perf_counter()
            codes = O.remap(hot, g)
            cold, codes = O.cold_plan(g, codes, mb.bag_ptr, nonpop, len(nonpop), bps, k_cap)
            stg = O.gather(table.array, cold)
            t2 = time.perf_counter()
            O.embbag_fwd(w.dtype, w_hot, k_cap, stg, codes, mb.bag_ptr, pop, len(pop), bps, mb.n_bags)
            O.embbag_fwd(w.dtype, w_hot, k_cap, stg, codes, mb.bag_ptr, nonpop, len(nonpop), bps, mb.n_bags)
            t3 = time.perf_counter()
            O.embbag_bwd_sgd(w.dtype, w_hot, k_cap, stg, codes, mb.bag_ptr, None, mb.n_samples, bps, dY, w.lr)
            t4 = time.perf_counter()
            t_all += t4 - t0
            for k, dt in zip(stage, (t1 - t0, t2 - t1, t3 - t2, t4 - t3)):
                stage[k] += dt
            L += mb.n_lookups
            B += mb.n_samples
            done += 1
    finally:
        os.sched_setaffinity(0, aff)
    log(f"[bench] cpu baseline: {done} batch steps in {t_all:.1f}s")
    mc = cpu_multicore_segregation(rows, hot, meas, min(3.0, budget_s))
    return {"value": L / t_all, "unit": "lookups/s", "cores": 1, "kind": "oracle",
            "multicore_segregation": mc,
            "classify_samples_per_s": B / stage["classify_partition"],
            "fwd_bwd_lookups_per_s": L / (stage["fwd"] + stage["bwd"]),
            "stage_ms_per_batch": {k: 1e3 * v / done for k, v in stage.items()},
            "sample": f"{done} batch steps of {w.name} (its {len(meas)} measured batches in turn), every per-batch "
                      f"step, single-threaded fp64 oracle pinned to host core {core}",
            "host_cpu": _cpu_model(), "host_nproc": os.cpu_count()}


def cpu_multicore_segregation(rows, hot, meas, budget_s):
    """Labelled multi-core CPU baseline, not the oracle: classify + partition of
    the same measured batches on the host's cores (OpenMP, at most 16 threads),
    the CPU-side segregation whose cost Sec. III measures.  The hot-set bitmap
    is built once, untimed (a learning phase's work); each batch is timed around
    the C call alone."""
    import ctypes as C
    import oracle as O

    n_rows = int(rows.sum(dtype=np.int64))
    bm, _ = O.mc_hot_bitmap(hot, n_rows)
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    L = O.mc_lib()
    rpt = np.ascontiguousarray(rows, dtype=np.uint32)
    nmax = max(mb.n_samples for mb in meas)
    flags = np.empty(nmax, dtype=np.uint8)
    pop = np.empty(nmax, dtype=np.int32)
    nonpop = np.empty(nmax, dtype=np.int32)
    ptr = lambda a: a.ctypes.data_as(C.c_void_p)
    calls = []
    for mb in meas:
        r = np.ascontiguousarray(mb.rows, dtype=np.uint32)
        bp = np.ascontiguousarray(mb.bag_ptr, dtype=np.int32)
        calls.append((r, bp, (len(rpt), ptr(rpt), ptr(r), ptr(bp), mb.n_samples, mb.bags_per_sample, ptr(bm),
                              threads, ptr(flags), ptr(pop), ptr(nonpop))))
    for _, _, a in calls[:2]:                       # thread team start-up, untimed
        L.mc_segregate(*a)
    t, done, S = 0.0, 0, 0
    while t < budget_s:
        _, _, a = calls[done % len(calls)]
        t0 = time.perf_counter()
        npop = L.mc_segregate(*a)
        t += time.perf_counter() - t0
        if npop < 0:
            raise SystemExit("multi-core segregation: bad argument")
        S += a[4]
        done += 1
    log(f"[bench] multi-core segregation: {done} batches on {threads} threads in {t:.2f}s")
    return {"value": S / t, "unit": "samples/s", "cores": threads, "kind": "openmp classify+partition, not the oracle",
            "us_per_batch": 1e6 * t / done,
            "sample": f"{done} classify+partition calls over the measured batches in turn, {threads} OpenMP threads"}


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


if __name__ == "__main__":
    main()
