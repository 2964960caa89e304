#!/usr/bin/env python3
"""Benchmark of the AVSG decode-step operator on one MI355X.

A step is one avsg_step over the whole batch: Stage One (hash matching, slot
reservation, MTP sharing, invalidation) and Stage Two (miss-only copy of host
rows into the reserved HBM slots).  The default workload is batch 64, top-K
2048, 8192 slots per request, two query tokens per step (MTP), 1,152-byte KV
rows plus 132-byte indexer-key rows in pinned host memory, step-to-step
retention 0.9.  Inputs for every step are generated and copied to HBM before
the timed region; the host rows stay in pinned host memory (they are what the
operator transfers).

Prints one JSON line.  `value` is microseconds per decode step (lower is
better); the line also carries the effective host-to-device bandwidth, the hit
rate, the roofline of the dominant kernel (the gather, bound by the host link)
and the CPU oracle timed on a sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PCIE_GEN5_X16_GBPS = 63.0   # 32 GT/s x 16 lanes x 128/130 / 8, one direction
METRIC = "µs per decode step for match+gather; effective H2D GB/s vs PCIe peak; hit rate"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=240)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--config", default="batch64_mtp2",
                    choices=["tiny", "batch16", "batch64_mtp2", "imbalance", "stress",
                             "stress_mtp3"])
    ap.add_argument("--gather", default="auto",
                    choices=["auto", "balanced", "request", "position", "sdma", "none", "pipelined", "resident",
                             "early"],
                    help="Stage Two (auto: resident reuse from 8192 lookups per step, else the paper's S3)")
    ap.add_argument("--match", default="hash", choices=["hash", "dualptr"])
    ap.add_argument("--workers", type=int, default=0, help="gather workgroups (0 = one per CU)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the pass that runs the timed steps from one captured HIP graph")
    ap.add_argument("--no-reference", action="store_true",
                    help="skip the reference run of the paper's Stage Two (every miss from the host)")
    ap.add_argument("--cpu-sample-steps", type=int, default=0,
                    help="oracle steps timed for the CPU baseline (0 = all warmup+timed steps)")
    ap.add_argument("--coherent", action="store_true", help="coherent (uncached) host rows")
    ap.add_argument("--report", default="", help="also write a detailed JSON report here")
    ap.add_argument("--appendix-d-sweep", default="",
                    help="run the S1/S2/S3 transfer sweep (batch x reuse) and write it here")
    ap.add_argument("--matching-sweep", default="",
                    help="run the Stage One latency sweeps (S=K=N, K at S=4096, S at K=512) and write them here")
    ap.add_argument("--lifetime-sweep", default="",
                    help="run the maximum-lifetime sweep (L = 1..32) and write it here")
    ap.add_argument("--config-table", default="",
                    help="run every workload under every Stage Two strategy (and the dual-pointer "
                         "ablation where it applies); write JSON rows here")
    ap.add_argument("--layer-batching", default="",
                    help="write the multi-layer batching comparison (one launch over every layer's tables "
                         "against one step per layer) to this JSON file and exit")
    ap.add_argument("--layers", type=int, default=8, help="layers of --layer-batching")
    ap.add_argument("--copy-engine-bench", default="",
                    help="copy-engine transfer of every workload in a process without torch, so the HIP "
                         "runtime's batched copy call is available; write JSON rows here")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-workload block (tiny, batch16, imbalance, stress) and the "
                         "multi-token cold-start reuse")
    ap.add_argument("--access-shape-probe", default="",
                    help="time the balanced gather on all-miss steps of three host layouts (1,152-byte KV "
                         "rows only, 132-byte indexer rows only, both) and write JSON rows here")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="run one device-to-device copy of this many MiB first (counter calibration)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this operator runs on one GPU; --gpus {args.gpus} is not supported "
              "(requests shard across GPUs with no communication, see the design notes)",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_engine_bench:
        copy_engine_bench(args.copy_engine_bench)
        return
    import torch
    import workload as W
    from paper_2609_37538_amd import avsg as A
    if args.appendix_d_sweep:
        appendix_d_sweep(args.appendix_d_sweep)
        return
    if args.matching_sweep:
        matching_sweep(args.matching_sweep)
        return
    if args.lifetime_sweep:
        lifetime_sweep(args.lifetime_sweep)
        return
    if args.config_table:
        config_table(args.config_table)
        return
    if args.layer_batching:
        layer_batching(args.layer_batching, args.layers)
        return
    if args.access_shape_probe:
        access_shape_probe(args.access_shape_probe)
        return

    gather_mode = {"balanced": A.AVSG_GATHER_BALANCED, "request": A.AVSG_GATHER_REQUEST,
                   "sdma": A.AVSG_GATHER_SDMA, "none": A.AVSG_GATHER_NONE,
                   "position": A.AVSG_GATHER_POSITION,
                   "pipelined": A.AVSG_GATHER_PIPELINED,
                   "resident": A.AVSG_GATHER_RESIDENT,
                   "early": A.AVSG_GATHER_EARLY, "auto": A.AVSG_GATHER_AUTO}[args.gather]
    match_mode = {"hash": A.AVSG_MATCH_HASH, "dualptr": A.AVSG_MATCH_DUALPTR}[args.match]
    spec = W.get_spec(args.config)
    if match_mode == A.AVSG_MATCH_DUALPTR:
        import dataclasses
        spec = dataclasses.replace(spec, slots=spec.topk)
    T = args.warmup + args.steps
    if spec.mode == "zipf_window" and T > spec.steps:
        raise SystemExit(f"{spec.name} defines {spec.steps} steps; warmup+steps = {T}")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    A.load()

    # ---- inputs: generated up front, copied to HBM before timing ----
    t_gen = time.time()
    wl = W.Workload(spec)
    X_host = wl.all_steps(T)                                   # [T][B][n_q][K] int32
    N_host = np.stack([wl.verified_len(t) for t in range(T)])  # [T][B] int64
    X_dev = torch.from_numpy(X_host).to(dev)
    N_dev = torch.from_numpy(N_host).to(dev)
    offs = wl.request_row_offsets()
    regions = []
    host_ptrs = []
    for s, rb in enumerate(spec.row_bytes):
        reg = A.HostRegion(wl.host_rows_total() * rb, coherent=args.coherent)
        W.fill_host(wl, s, reg.ptr)
        regions.append(reg)
        host_ptrs += [reg.ptr + int(offs[r]) * rb for r in range(spec.batch)]
    gen_s = time.time() - t_gen

    cfg = A.make_config(spec.batch, spec.topk, spec.n_q, spec.slots, row_bytes=spec.row_bytes,
                        gather_workers=args.workers, match_mode=match_mode, gather_mode=gather_mode)
    # the transfer the library runs for this configuration (auto resolved)
    gather_mode = A.avsg_resolve_config(cfg).gather_mode
    gather_name = {A.AVSG_GATHER_BALANCED: "balanced", A.AVSG_GATHER_REQUEST: "request",
                   A.AVSG_GATHER_SDMA: "sdma", A.AVSG_GATHER_NONE: "none", A.AVSG_GATHER_POSITION: "position",
                   A.AVSG_GATHER_PIPELINED: "pipelined", A.AVSG_GATHER_RESIDENT: "resident",
                   A.AVSG_GATHER_EARLY: "early"}[gather_mode]
    stream = torch.cuda.current_stream(dev)
    op = A.Operator(cfg, host_ptrs, wl.ctx, device=dev, stream=stream)

    # ---- measured hipMemcpy H2D peak (pinned host -> HBM, 512 MiB) ----
    peak_bytes = min(512 << 20, regions[0].nbytes)
    tmp = torch.empty(peak_bytes, dtype=torch.uint8, device=dev)
    memcpy_peak = A.avsg_h2d_peak(regions[0].ptr, tmp.data_ptr(), peak_bytes, 20, stream.cuda_stream)
    del tmp

    if args.copy_probe_mib > 0:
        a = torch.ones(args.copy_probe_mib << 20, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    # ---- warmup, then the timed region (HIP events on the step stream from
    # step 0, so the cold start is reported on its own) ----
    A.avsg_set_timing(op.h, True)
    for t in range(args.warmup):
        op.step(X_dev[t], N_dev[t] if spec.speculative else None)
    torch.cuda.synchronize()
    before = op.stats()
    before_r = [op.request_stats(r) for r in range(spec.batch)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(args.warmup, T):
        op.step(X_dev[t], N_dev[t] if spec.speculative else None)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    match_all, gather_all, tail_all = A.avsg_timing(op.h, T)
    A.avsg_set_timing(op.h, False)
    after = op.stats()
    after_r = [op.request_stats(r) for r in range(spec.batch)]
    # request-averaged hit rate over the timed steps (each request's own rate, then the mean)
    per_req = [(a["hits"] - b["hits"]) / max(1, a["lookups"] - b["lookups"]) for a, b in zip(after_r, before_r)]
    match_ms, gather_ms = match_all[args.warmup:], gather_all[args.warmup:]
    tail_ms = tail_all[args.warmup:]
    wall_events = wall

    # ---- the same steps from a cold start on a fresh operator without the
    # per-kernel events: the step rate a caller sees (`value`) ----
    op_plain = A.Operator(cfg, host_ptrs, wl.ctx, device=dev, stream=stream)
    for t in range(args.warmup):
        op_plain.step(X_dev[t], N_dev[t] if spec.speculative else None)
    torch.cuda.synchronize()
    plain_before = op_plain.stats()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(args.warmup, T):
        op_plain.step(X_dev[t], N_dev[t] if spec.speculative else None)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    plain_after = op_plain.stats()
    op_plain.close()
    for k in ("hits", "misses", "host_bytes"):
        if plain_after[k] - plain_before[k] != after[k] - before[k]:
            raise RuntimeError(f"the uninstrumented pass differs from the timed pass in {k}")

    # ---- the same steps executed from a HIP graph: after the warmup, the
    # timed steps (each one's selections copied into one input buffer, then
    # avsg_step on it) are captured on a fresh operator as a single graph and
    # replayed once, so no per-launch host work remains in the timed region ----
    graph = None
    if (not args.no_graph and match_mode == A.AVSG_MATCH_HASH
            and gather_mode not in (A.AVSG_GATHER_SDMA, A.AVSG_GATHER_NONE)):
        op_g = A.Operator(cfg, host_ptrs, wl.ctx, device=dev, stream=torch.cuda.Stream(dev))
        for t in range(args.warmup):
            op_g.step(X_dev[t], N_dev[t] if spec.speculative else None)
        X_in = torch.empty_like(X_dev[0])
        N_in = torch.empty_like(N_dev[0])
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=op_g.stream):
            for t in range(args.warmup, T):
                X_in.copy_(X_dev[t])
                if spec.speculative:
                    N_in.copy_(N_dev[t])
                op_g.step(X_in, N_in if spec.speculative else None)
        torch.cuda.synchronize()
        g_before = op_g.stats()
        t0 = time.perf_counter()
        g.replay()
        torch.cuda.synchronize()
        wall_g = time.perf_counter() - t0
        g_after = op_g.stats()
        del g
        op_g.close()
        for k in ("hits", "misses", "host_bytes"):
            if g_after[k] - g_before[k] != after[k] - before[k]:
                raise RuntimeError(f"the graph-executed pass differs from the timed pass in {k}")
        graph = {"value": round(wall_g / args.steps * 1e6, 2), "unit": "us/step",
                 "what": "the timed steps captured as one HIP graph (each step's selections "
                         "copied into the captured input, then avsg_step) and replayed once"}

    # ---- reference: the paper's Stage Two (S3, every miss copied from the
    # host) on the same steps, same host rows, same stream ----
    reference = None
    if gather_mode in (A.AVSG_GATHER_RESIDENT, A.AVSG_GATHER_EARLY) and not args.no_reference:
        cfg_ref = A.make_config(spec.batch, spec.topk, spec.n_q, spec.slots, row_bytes=spec.row_bytes,
                                gather_workers=args.workers, match_mode=match_mode,
                                gather_mode=A.AVSG_GATHER_BALANCED)
        op_ref = A.Operator(cfg_ref, host_ptrs, wl.ctx, device=dev, stream=stream)
        for t in range(args.warmup):
            op_ref.step(X_dev[t], N_dev[t] if spec.speculative else None)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for t in range(args.warmup, T):
            op_ref.step(X_dev[t], N_dev[t] if spec.speculative else None)
        torch.cuda.synchronize()
        wall_ref = time.perf_counter() - t1
        # the same steps once more from a cold start with HIP events around
        # each kernel: the S3 gather kernel's own duration and bandwidth
        op_ref.close()
        op_ref = A.Operator(cfg_ref, host_ptrs, wl.ctx, device=dev, stream=stream)
        for t in range(args.warmup):
            op_ref.step(X_dev[t], N_dev[t] if spec.speculative else None)
        torch.cuda.synchronize()
        ref_before = op_ref.stats()
        A.avsg_set_timing(op_ref.h, True)
        for t in range(args.warmup, T):
            op_ref.step(X_dev[t], N_dev[t] if spec.speculative else None)
        ref_match_ms, ref_gather_ms, _ = A.avsg_timing(op_ref.h, args.steps)
        ref_after = op_ref.stats()
        op_ref.close()
        ref_host = ref_after["host_bytes"] - ref_before["host_bytes"]
        ref_gsec = float(np.sum(ref_gather_ms)) * 1e-3
        ref_gbps = ref_host / ref_gsec / 1e9 if ref_gsec > 0 else 0.0
        s3_block = (_traffic_block(TRAFFIC_SUMMARY_S3)
                    if (args.config, args.workers, args.match) == ("batch64_mtp2", 0, "hash") else None)
        reference = {"gather": "balanced", "value": round(wall_ref / args.steps * 1e6, 2),
                     "unit": "us/step",
                     "what": "the paper's Stage Two (S3, Eq. 6): every miss copied from the host",
                     "match_us_median": round(float(np.median(ref_match_ms)) * 1e3, 2),
                     "gather_us_median": round(float(np.median(ref_gather_ms)) * 1e3, 2),
                     "roofline": {"bound": "pcie", "kernel": "gather_balanced_kernel",
                                  "achieved": round(ref_gbps, 3), "peak": PCIE_GEN5_X16_GBPS, "unit": "GB/s",
                                  "frac": round(ref_gbps / PCIE_GEN5_X16_GBPS, 4),
                                  "frac_of_hipmemcpy_peak": round(ref_gbps / memcpy_peak, 4) if memcpy_peak else None,
                                  "algorithmic_bytes_per_launch": round(ref_host / args.steps),
                                  "traffic": None, "traffic_source": None,
                                  "what": "every miss's row bytes over the host link / the S3 kernel's "
                                          "average duration (HIP events on the step stream)"}}
        if s3_block:
            reference["roofline"]["traffic"] = s3_block["traffic_bytes_per_launch"]
            reference["roofline"]["traffic_source"] = TRAFFIC_SUMMARY_S3
            reference["roofline"]["traffic_over_algorithmic"] = round(
                s3_block["traffic_bytes_per_launch"] / s3_block["algorithmic_traffic_bytes_per_launch"], 3)
            # what the host link itself carried (128-byte lines, per the
            # counters): a row that several tokens of a step miss is read over
            # the link once and served from L2 after, so `achieved` (every
            # miss's row) can exceed what the link moves
            link_gbps = s3_block["host_read_bytes_per_launch"] * args.steps / ref_gsec / 1e9 if ref_gsec else 0.0
            reference["roofline"]["host_link_bytes_per_launch"] = s3_block["host_read_bytes_per_launch"]
            reference["roofline"]["host_link_gbps"] = round(link_gbps, 3)
            reference["roofline"]["host_link_frac"] = round(link_gbps / PCIE_GEN5_X16_GBPS, 4)

    K = args.steps
    us_per_step = wall / K * 1e6
    lookups = after["lookups"] - before["lookups"]
    hits = after["hits"] - before["hits"]
    misses = after["misses"] - before["misses"]
    row_total = sum(spec.row_bytes)
    moved = misses * row_total if gather_mode != A.AVSG_GATHER_NONE else 0
    host_moved = after["host_bytes"] - before["host_bytes"]
    pipelined = gather_mode == A.AVSG_GATHER_PIPELINED
    early = gather_mode == A.AVSG_GATHER_EARLY
    early_info = None
    if early:
        # three launches: the early list (timed in the matching slot), Stage
        # One beside the early copies (the main Stage Two slot) and the
        # finishing kernel (the tail slot); matching runs inside the second
        early_info = {
            "early_list_us_median": round(float(np.median(match_ms)) * 1e3, 2) if len(match_ms) else None,
            "match_and_early_copy_us_median": round(float(np.median(gather_ms)) * 1e3, 2) if len(gather_ms) else None,
            "finish_us_median": round(float(np.median(tail_ms)) * 1e3, 2) if len(tail_ms) else None,
            "early_rows_per_step": round((after["early_rows"] - before["early_rows"]) / args.steps, 1),
            "early_staged_rows_per_step": round((after["early_staged_rows"] - before["early_staged_rows"])
                                                / args.steps, 1),
            "early_deferred_rows_per_step": round((after["early_deferred_rows"]
                                                   - before["early_deferred_rows"]) / args.steps, 1),
        }
    if pipelined:
        # one fused launch: its duration is recorded in the matching slot
        gather_ms, match_ms = match_ms, np.zeros_like(match_ms)
        gather_all, match_all = match_all, np.zeros_like(match_all)
    n_step = min(len(match_ms), len(gather_ms))
    step_ms = (np.nan_to_num(np.asarray(match_ms[:n_step], dtype=np.float64))
               + np.nan_to_num(np.asarray(gather_ms[:n_step], dtype=np.float64)))
    if len(tail_ms) >= n_step:
        step_ms = step_ms + np.nan_to_num(np.asarray(tail_ms[:n_step], dtype=np.float64))
    gather_s = float(np.sum(gather_ms)) * 1e-3
    match_s = float(np.sum(match_ms)) * 1e-3
    gather_gbps = host_moved / gather_s / 1e9 if gather_s > 0 and host_moved else 0.0
    eff_gbps = host_moved / wall / 1e9 if host_moved else 0.0

    # ---- CPU baseline: the oracle on the same inputs ----
    cpu = None
    if not args.no_cpu_baseline and match_mode == A.AVSG_MATCH_HASH:
        cpu = cpu_baseline(spec, wl, X_host, N_host, host_ptrs, args, gather_mode)

    traffic = measured_traffic(args, gather_name)
    configs = None
    cold = None
    if not args.no_configs and args.config == "batch64_mtp2" and gather_name == "resident" \
            and args.match == "hash":
        configs = {"batch64_mtp2": {
            "transfer": gather_name,
            "us_per_step": round(us_per_step, 2),
            "match_us_median": round(float(np.median(match_ms)) * 1e3, 2),
            "stage_two_us_median": round(float(np.median(gather_ms)) * 1e3, 2),
            "h2d_gbps_gather_kernel": round(gather_gbps, 3),
            "frac_of_hipmemcpy_peak": round(gather_gbps / memcpy_peak, 4) if memcpy_peak else None,
            "frac_of_pcie_gen5_x16": round(gather_gbps / PCIE_GEN5_X16_GBPS, 4),
            "hit_rate": round(hits / max(1, lookups), 5),
            "s3_us_per_step": reference["value"] if reference else None,
            "s3_gbps_gather_kernel": reference["roofline"]["achieved"] if reference else None,
            "s3_frac_of_hipmemcpy_peak": reference["roofline"]["frac_of_hipmemcpy_peak"] if reference else None,
            "cpu_oracle_us_per_step": cpu["value"] if cpu else None,
            "cpu_oracle_threads": cpu["cores"] if cpu else None,
            "steps_timed": f"{args.warmup}..{T - 1}"}}
        for reg in regions:
            reg.free()
        regions = []
        configs.update(config_block(memcpy_peak, dev, with_cpu=not args.no_cpu_baseline))
        cold = mtp_cold_start_reuse(dev)
    out = {
        "metric": METRIC,
        "value": round(us_per_step, 2),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(us_per_step / 1e3, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {
            "workload": spec.name, "batch": spec.batch, "topk": spec.topk, "slots": spec.slots,
            "n_q": spec.n_q, "context": int(wl.ctx.max()), "row_bytes": list(spec.row_bytes),
            "retention": spec.retention, "match": args.match,
            "gather": gather_name if args.gather == gather_name else f"{args.gather} ({gather_name})",
            "steps_timed": f"{args.warmup}..{T - 1}",
        },
        "hit_rate": round(hits / max(1, lookups), 5),
        "hit_rate_request_mean": round(float(np.mean(per_req)), 5),
        "hit_rate_from_step0": round(after["hits"] / max(1, after["lookups"]), 5),
        "lost_installs_per_step": round((after["lost_exhausted"] + after["lost_collision"]
                                         - before["lost_exhausted"] - before["lost_collision"]) / K, 1),
        "misses_per_step": round(misses / K, 1),
        "host_rows_per_step": round(host_moved / row_total / K, 1) if row_total else 0.0,
        # resident reuse: misses filled from another slot of the request, and
        # same-step repeats (written by their index's host copy or copied after)
        "resident_rows_per_step": round((after["resident_rows"] - before["resident_rows"]) / K, 1),
        "repeat_rows_per_step": round((after["duplicate_rows"] - before["duplicate_rows"]) / K, 1),
        "delivered_gbps": round(moved / wall / 1e9, 3) if moved else 0.0,
        "h2d_gbps_effective": round(eff_gbps, 3),
        "h2d_gbps_gather_kernel": round(gather_gbps, 3),
        "hipmemcpy_h2d_peak_gbps": round(memcpy_peak, 3),
        "frac_of_hipmemcpy_peak": round(gather_gbps / memcpy_peak, 4) if memcpy_peak else None,
        "frac_of_pcie_gen5_x16": round(gather_gbps / PCIE_GEN5_X16_GBPS, 4),
        "match_us_median": (round(float(np.median(match_ms)) * 1e3, 2)
                            if len(match_ms) and not pipelined else None),
        "gather_us_median": round(float(np.median(gather_ms)) * 1e3, 2) if len(gather_ms) else None,
        "repeat_copy_us_median": (round(float(np.median(tail_ms)) * 1e3, 2)
                                  if gather_mode == A.AVSG_GATHER_RESIDENT and len(tail_ms) else None),
        "early_fetch": early_info,
        "match_us_p99": (round(float(np.percentile(match_ms, 99)) * 1e3, 2)
                         if len(match_ms) and not pipelined else None),
        "gather_us_p99": round(float(np.percentile(gather_ms, 99)) * 1e3, 2) if len(gather_ms) else None,
        # every kernel of a step (matching, Stage Two, repeat or finishing kernel) summed per step
        "step_kernels_us_median": (round(float(np.median(step_ms)) * 1e3, 2) if len(step_ms) else None),
        "step_kernels_us_p99": (round(float(np.percentile(step_ms, 99)) * 1e3, 2) if len(step_ms) else None),
        "cold_start_step0_us": ({"match": None if pipelined else round(float(match_all[0]) * 1e3, 2),
                                 "gather": round(float(gather_all[0]) * 1e3, 2)}
                                if len(gather_all) == T else None),
        "match_frac_of_step": round(match_s / wall_events, 4),
        "us_per_step_with_kernel_events": round(wall_events / K * 1e6, 2),
        "roofline": {
            "bound": "pcie",
            "kernel": {"balanced": "gather_balanced_kernel", "resident": "gather_resident_kernel",
                       "pipelined": "step_pipelined_kernel",
                       "early": "step_early_kernel"}.get(gather_name, gather_name),
            "achieved": round(gather_gbps, 3),
            "peak": PCIE_GEN5_X16_GBPS,
            "unit": "GB/s",
            "frac": round(gather_gbps / PCIE_GEN5_X16_GBPS, 4),
            "traffic": traffic["traffic_bytes_per_launch"] if traffic else None,
            "traffic_source": TRAFFIC_SUMMARY if traffic else None,
            # same basis as `traffic`: host-link reads + HBM reads (resident
            # sources) + HBM writes (host, fan and resident rows)
            "algorithmic_traffic_bytes_per_launch": (traffic.get("algorithmic_traffic_bytes_per_launch")
                                                     if traffic else None),
            "traffic_over_algorithmic": (round(traffic["traffic_bytes_per_launch"]
                                               / traffic["algorithmic_traffic_bytes_per_launch"], 3)
                                         if traffic and traffic.get("algorithmic_traffic_bytes_per_launch")
                                         else None),
            "algorithmic_bytes_per_launch": round(host_moved / K) if host_moved else 0,
            # what the host link itself carried per launch (128-byte lines,
            # per the counters) and its rate over the same launches
            "host_link_bytes_per_launch": traffic.get("host_read_bytes_per_launch") if traffic else None,
            "host_link_gbps": (round(traffic["host_read_bytes_per_launch"] * K / gather_s / 1e9, 3)
                               if traffic and gather_s > 0 else None),
            "measured_hipmemcpy_peak": round(memcpy_peak, 3),
        },
        "cpu_baseline": cpu,
        "graph_replay": graph,
        "reference_all_misses_from_host": reference,
        "configs": configs,
        "mtp_cold_start_reuse": cold,
    }
    print(json.dumps(out), flush=True)
    if args.report:
        rep = dict(out)
        rep["gen_seconds"] = round(gen_s, 1)
        rep["match_ms"] = [round(float(x), 4) for x in match_ms]
        rep["gather_ms"] = [round(float(x), 4) for x in gather_ms]
        rep["stats"] = after
        with open(args.report, "w") as f:
            json.dump(rep, f, indent=1)
    op.close()
    for reg in regions:
        reg.free()


def _fill_regions(spec, wl):
    """Pinned host regions of every stream, filled with the workload's rows;
    returns (regions, row pointers ordered s*B + r)."""
    import workload as W
    from paper_2609_37538_amd import avsg as A
    offs = wl.request_row_offsets()
    regions, ptrs = [], []
    for s, rb in enumerate(spec.row_bytes):
        reg = A.HostRegion(wl.host_rows_total() * rb)
        W.fill_host(wl, s, reg.ptr)
        regions.append(reg)
        ptrs += [reg.ptr + int(offs[r]) * rb for r in range(spec.batch)]
    return regions, ptrs


def _measure(spec, gather_mode, X, N, ptrs, ctx, warm, timed, dev):
    """One Stage Two mode on prepared inputs: a pass without per-kernel events
    (wall time per step, as a caller sees it) and a pass with HIP events
    around each kernel, each on a fresh operator from the same cold start;
    both must move the same rows."""
    import torch
    from paper_2609_37538_amd import avsg as A
    cfg = A.make_config(spec.batch, spec.topk, spec.n_q, spec.slots, row_bytes=spec.row_bytes,
                        gather_mode=gather_mode)
    res = {}
    for events in (False, True):
        op = A.Operator(cfg, ptrs, ctx, device=dev)
        try:
            for t in range(warm):
                op.step(X[t], N[t] if N is not None else None)
            torch.cuda.synchronize()
            before = op.stats()
            if events:
                A.avsg_set_timing(op.h, True)
            t0 = time.perf_counter()
            for t in range(warm, warm + timed):
                op.step(X[t], N[t] if N is not None else None)
            torch.cuda.synchronize()
            wall = time.perf_counter() - t0
            if events:
                match_ms, gather_ms, tail_ms = A.avsg_timing(op.h, timed)
            after = op.stats()
        finally:
            op.close()
        d = {k: after[k] - before[k] for k in ("hits", "lookups", "misses", "host_bytes")}
        if events:
            if d != res["delta"]:
                raise RuntimeError(f"{spec.name}: the timed pass with events differs from the plain pass")
            stage_two = np.asarray(gather_ms, dtype=np.float64) + np.asarray(tail_ms, dtype=np.float64)
            res["match_ms"], res["stage_two_ms"] = np.asarray(match_ms, dtype=np.float64), stage_two
        else:
            res["wall"], res["delta"] = wall, d
    return res


def config_block(memcpy_peak, dev, warm=8, timed=32, with_cpu=True):
    """The other benchmark workloads (tiny, batch16, imbalance, stress) at full
    size, each from a cold start: `warm` untimed steps, then `timed` steps under
    the default Stage Two (AVSG_GATHER_AUTO: resident reuse from 8192 lookups per
    step, else S3; `transfer` names it), under the paper's S3, under resident
    reuse where that is not the default, and on the imbalance mix under the
    request-level S1 it is compared with.  Per workload:
    µs per step (wall time between two synchronizations, no per-kernel events),
    matching and Stage Two kernel medians (HIP events), host-link payload GB/s
    of the Stage Two kernels and its fractions of the measured hipMemcpy H2D
    peak and of PCIe Gen5 x16, hit rate, and the CPU oracle on the same steps."""
    import torch
    import workload as W
    from paper_2609_37538_amd import avsg as A
    out = {}
    for name in ("tiny", "batch16", "imbalance", "stress"):
        t_start = time.time()
        spec = W.get_spec(name)
        wl = W.Workload(spec)
        X_host = wl.all_steps(warm + timed)
        N_host = np.stack([wl.verified_len(t) for t in range(warm + timed)])
        X = torch.from_numpy(X_host).to(dev)
        N = torch.from_numpy(N_host).to(dev) if spec.speculative else None
        regions, ptrs = _fill_regions(spec, wl)
        row_total = sum(spec.row_bytes)
        entry = {"batch": spec.batch, "topk": spec.topk, "slots": spec.slots, "n_q": spec.n_q,
                 "context": int(wl.ctx.max()), "row_bytes": list(spec.row_bytes),
                 "steps_timed": f"{warm}..{warm + timed - 1}"}
        auto = A.avsg_resolve_config(A.make_config(spec.batch, spec.topk, spec.n_q, spec.slots,
                                                   row_bytes=spec.row_bytes,
                                                   gather_mode=A.AVSG_GATHER_AUTO)).gather_mode
        entry["transfer"] = "resident" if auto == A.AVSG_GATHER_RESIDENT else "s3"
        modes = [("default", A.AVSG_GATHER_AUTO), ("s3", A.AVSG_GATHER_BALANCED)]
        if auto != A.AVSG_GATHER_RESIDENT:
            modes.append(("resident", A.AVSG_GATHER_RESIDENT))
        if name == "imbalance":
            modes.append(("s1", A.AVSG_GATHER_REQUEST))
        try:
            for label, gm in modes:
                m = _measure(spec, gm, X, N, ptrs, wl.ctx, warm, timed, dev)
                d = m["delta"]
                gsec = float(np.sum(m["stage_two_ms"])) * 1e-3
                gbps = d["host_bytes"] / gsec / 1e9 if gsec > 0 and d["host_bytes"] else 0.0
                pre = "" if label == "default" else label + "_"
                entry[pre + "us_per_step"] = round(m["wall"] / timed * 1e6, 2)
                entry[pre + "match_us_median"] = round(float(np.median(m["match_ms"])) * 1e3, 2)
                entry[pre + "stage_two_us_median"] = round(float(np.median(m["stage_two_ms"])) * 1e3, 2)
                entry[pre + "h2d_gbps_gather_kernel"] = round(gbps, 3)
                entry[pre + "frac_of_hipmemcpy_peak"] = round(gbps / memcpy_peak, 4) if memcpy_peak else None
                entry[pre + "frac_of_pcie_gen5_x16"] = round(gbps / PCIE_GEN5_X16_GBPS, 4)
                if label == "default":
                    entry["hit_rate"] = round(d["hits"] / max(1, d["lookups"]), 5)
                    entry["misses_per_step"] = round(d["misses"] / timed, 1)
                    entry["host_rows_per_step"] = round(d["host_bytes"] / row_total / timed, 1)
                    entry["match_frac_of_step"] = round(float(np.sum(m["match_ms"])) * 1e-3 / m["wall"], 4)
            if with_cpu:
                us, threads = _oracle_us_per_step(spec, X_host, N_host, ptrs, warm, timed)
                entry["cpu_oracle_us_per_step"] = round(us, 1)
                entry["cpu_oracle_threads"] = threads
        finally:
            for reg in regions:
                reg.free()
        entry["seconds"] = round(time.time() - t_start, 1)
        out[name] = entry
        print(json.dumps({"config": name, **entry}), file=sys.stderr, flush=True)
    return out


def mtp_cold_start_reuse(dev):
    """Reuse at the cold start (step 0 of an empty table) with N_q = 1..4 query
    tokens per request: one table shared by a request's tokens (later tokens
    hit the slots earlier tokens reserved) against one independent table per
    token (no index of a token can hit at step 0).  Matching only, on the
    token mixes of batch64_mtp2 (token g >= 1 keeps 95% of token 0's indices)
    and of stress (recency window shifted per token, 95% of the hot set kept).
    reuse = hits / (B * N_q * K) at step 0."""
    import dataclasses
    import torch
    import workload as W
    from paper_2609_37538_amd import avsg as A
    host = A.HostRegion(1 << 16)
    out = {}
    try:
        for mix in ("batch64_mtp2", "stress"):
            rows = {}
            for n_q in (1, 2, 3, 4):
                spec = dataclasses.replace(W.get_spec(mix), n_q=n_q)
                wl = W.Workload(spec)
                X = wl.topk(0)
                B, K = spec.batch, spec.topk
                res = {}
                for label, (b, nq, Xs) in (("shared", (B, n_q, X)),
                                            ("independent", (B * n_q, 1, X.reshape(B * n_q, 1, K)))):
                    cfg = A.make_config(b, K, nq, spec.slots, row_bytes=(16,), gather_mode=A.AVSG_GATHER_NONE)
                    ctx = np.repeat(wl.ctx, n_q) if label == "independent" else wl.ctx
                    op = A.Operator(cfg, [host.ptr] * b, ctx, device=dev)
                    try:
                        op.step(torch.from_numpy(np.ascontiguousarray(Xs)).to(dev))
                        st = op.stats()
                    finally:
                        op.close()
                    res[label] = round(st["hits"] / max(1, st["lookups"]), 5)
                    if label == "shared":
                        res["lost_installs"] = int(st["lost_exhausted"] + st["lost_collision"])
                rows[str(n_q)] = res
            out[mix] = rows
    finally:
        host.free()
    return out


def access_shape_probe(out_path, warm=4, timed=16):
    """The balanced gather (S3) on steps where nearly every selected index
    misses (retention 0 over 1M-token contexts), for three host layouts: 1,152-
    byte KV rows only (nine whole 128-byte lines per row), 132-byte indexer
    rows only (two lines per row), and both regions (the batch64_mtp2 layout:
    eleven lines per token).  Reports payload GB/s and line GB/s (bytes of the
    128-byte lines the rows touch) of the gather kernel, from HIP events on
    the step stream, beside the measured hipMemcpy H2D peak."""
    import torch
    import workload as W
    from paper_2609_37538_amd import avsg as A
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    probe = A.HostRegion(512 << 20)
    tmp = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    peak = A.avsg_h2d_peak(probe.ptr, tmp.data_ptr(), 512 << 20, 20, torch.cuda.current_stream(dev).cuda_stream)
    del tmp
    probe.free()
    results = [{"hipmemcpy_h2d_peak_gbps": round(peak, 3)}]
    print(json.dumps(results[0]), flush=True)

    def lines(rb):
        # rows of rb bytes at offsets x * rb from a 4 KiB-aligned base
        if rb % 128 == 0:
            return rb // 128
        return 2 if rb == 132 else -1

    for label, row_bytes in (("kv_1152", (W.KV_ROW_BYTES,)), ("indexer_132", (W.INDEXER_ROW_BYTES,)),
                             ("kv_and_indexer", (W.KV_ROW_BYTES, W.INDEXER_ROW_BYTES))):
        spec = W.custom_spec(name=f"shape_{label}", cfg_id=12, batch=16, topk=2048, slots=8192, n_q=1,
                             steps=warm + timed, ctx=1 << 20, retention=0.0, row_bytes=row_bytes)
        wl = W.Workload(spec)
        X = torch.from_numpy(wl.all_steps(warm + timed)).to(dev)
        regions, ptrs = _fill_regions(spec, wl)
        try:
            m = _measure(spec, A.AVSG_GATHER_BALANCED, X, None, ptrs, wl.ctx, warm, timed, dev)
        finally:
            for reg in regions:
                reg.free()
        d = m["delta"]
        gsec = float(np.sum(m["stage_two_ms"])) * 1e-3
        misses = d["misses"]
        line_bytes = misses * 128 * sum(lines(rb) for rb in row_bytes)
        row = {"layout": label, "row_bytes": list(row_bytes), "batch": 16, "topk": 2048,
               "misses_per_step": round(misses / timed, 1),
               "gather_us_median": round(float(np.median(m["stage_two_ms"])) * 1e3, 2),
               "payload_gbps": round(d["host_bytes"] / gsec / 1e9, 3),
               "line_gbps": round(line_bytes / gsec / 1e9, 3),
               "line_frac_of_hipmemcpy_peak": round(line_bytes / gsec / 1e9 / peak, 4)}
        results.append(row)
        print(json.dumps(row), flush=True)
    with open(out_path, "w") as f:
        json.dump(results, f, indent=1)


def appendix_d_sweep(out_path):
    """Transfer efficiency of the three core-binding strategies (request-level
    S1, equal top-K positions S2, balanced miss list S3) over batch sizes
    {1,2,4,8,16,32} and reuse {0, .25, .5, .75, 1}, K = 2048, one query token,
    1,152-byte rows.  Reuse is controlled by a fixed hot set selected every step
    plus never-seen ids; each point runs 8 warm-up steps then times 16 steps.
    Effective bandwidth = moved bytes / summed Stage Two kernel time."""
    import torch
    import workload as W
    from paper_2609_37538_amd import avsg as A
    Bs, reuses = [1, 2, 4, 8, 16, 32], [0.0, 0.25, 0.5, 0.75, 1.0]
    modes = [("S1", A.AVSG_GATHER_REQUEST), ("S2", A.AVSG_GATHER_POSITION),
             ("S3", A.AVSG_GATHER_BALANCED)]
    K, S, ctx, warm, timed = 2048, 8192, 65536, 8, 16
    dev = torch.device("cuda:0")
    base = W.custom_spec(name="appendix_d", cfg_id=10, batch=max(Bs), topk=K, slots=S, n_q=1,
                         steps=warm + timed, ctx=ctx, mode="controlled")
    host = A.HostRegion(max(Bs) * ctx * W.KV_ROW_BYTES)
    W.fill_host(W.Workload(base), 0, host.ptr)
    results = []
    for B in Bs:
        for reuse in reuses:
            import dataclasses
            spec = dataclasses.replace(base, batch=B, retention=reuse)
            wl = W.Workload(spec)
            X = torch.from_numpy(wl.all_steps(warm + timed)).to(dev)
            ptrs = [host.ptr + r * ctx * W.KV_ROW_BYTES for r in range(B)]
            for name, mode in modes:
                cfg = A.make_config(B, K, 1, S, row_bytes=(W.KV_ROW_BYTES,), gather_mode=mode)
                op = A.Operator(cfg, ptrs, wl.ctx, device=dev)
                for t in range(warm):
                    op.step(X[t])
                torch.cuda.synchronize()
                before = op.stats()
                A.avsg_set_timing(op.h, True)
                for t in range(warm, warm + timed):
                    op.step(X[t])
                _, gather_ms, _ = A.avsg_timing(op.h, timed)
                after = op.stats()
                op.close()
                misses = after["misses"] - before["misses"]
                moved = misses * W.KV_ROW_BYTES
                gsec = float(np.sum(gather_ms)) * 1e-3
                row = {"batch": B, "reuse_target": reuse, "strategy": name,
                       "hit_rate": round((after["hits"] - before["hits"]) /
                                         max(1, after["lookups"] - before["lookups"]), 4),
                       "misses_per_step": round(misses / timed, 1),
                       "gather_us": round(gsec / timed * 1e6, 2),
                       "gbps": round(moved / gsec / 1e9, 3) if gsec > 0 else 0.0}
                results.append(row)
                print(json.dumps(row), flush=True)
    host.free()
    with open(out_path, "w") as f:
        json.dump(results, f, indent=1)


def _timed_run(spec, cfg_kw, warm, timed, host_ptrs, dev, verified=False):
    """Run warm + timed steps of `spec` through one operator; return
    (match_ms[], gather_ms[], stats delta, wall seconds of the timed steps)."""
    import torch
    import workload as W
    from paper_2609_37538_amd import avsg as A
    wl = W.Workload(spec)
    X = torch.from_numpy(wl.all_steps(warm + timed)).to(dev)
    N = torch.from_numpy(np.stack([wl.verified_len(t) for t in range(warm + timed)])).to(dev)
    cfg = A.make_config(spec.batch, spec.topk, spec.n_q, spec.slots, **cfg_kw)
    op = A.Operator(cfg, host_ptrs, wl.ctx, device=dev)
    try:
        for t in range(warm):
            op.step(X[t], N[t] if verified else None)
        torch.cuda.synchronize()
        before = op.stats()
        A.avsg_set_timing(op.h, True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for t in range(warm, warm + timed):
            op.step(X[t], N[t] if verified else None)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        match_ms, gather_ms, tail_ms = A.avsg_timing(op.h, timed)
        gather_ms = gather_ms + tail_ms       # all of Stage Two
        after = op.stats()
    finally:
        op.close()
    delta = {k: after[k] - before[k] for k in after if k != "max_step_alloc_decays"}
    return match_ms, gather_ms, delta, wall


def layer_batching(out_path, layers, warm=16, timed=64):
    """Multi-layer batching: the 64 tables of batch64_mtp2 read as `layers`
    layers of 64 / layers requests (every (layer, request) pair has its own
    table, buffer and host rows).  A decode step is either one launch over
    every pair (possible when all layers' selections are known together) or
    one step per layer in sequence (in a model, a layer's selection waits for
    the previous layer's attention).  Same selections, host rows and stream;
    slots, counts and buffers must agree byte for byte."""
    import torch
    import workload as W
    from paper_2609_37538_amd import avsg as A
    spec = W.get_spec("batch64_mtp2")
    B = spec.batch
    if layers < 1 or B % layers:
        raise SystemExit(f"--layers must divide {B}")
    per = B // layers
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = W.Workload(spec)
    X = torch.from_numpy(wl.all_steps(warm + timed)).to(dev)
    offs = wl.request_row_offsets()
    regions, ptrs = [], []
    for s, rb in enumerate(spec.row_bytes):
        reg = A.HostRegion(wl.host_rows_total() * rb)
        W.fill_host(wl, s, reg.ptr)
        regions.append(reg)
        ptrs += [reg.ptr + int(offs[r]) * rb for r in range(B)]
    ns = len(spec.row_bytes)
    results = []
    for name, gm in (("resident reuse", A.AVSG_GATHER_RESIDENT), ("early fetch", A.AVSG_GATHER_EARLY),
                     ("S3 balanced", A.AVSG_GATHER_BALANCED), ("pipelined", A.AVSG_GATHER_PIPELINED)):
        kw = dict(row_bytes=spec.row_bytes, gather_mode=gm)
        one = A.Operator(A.make_config(B, spec.topk, spec.n_q, spec.slots, **kw), ptrs, wl.ctx, device=dev)
        each = [A.Operator(A.make_config(per, spec.topk, spec.n_q, spec.slots, **kw),
                           [ptrs[s * B + l * per + i] for s in range(ns) for i in range(per)],
                           wl.ctx[l * per:(l + 1) * per], device=dev)
                for l in range(layers)]
        walls = {}
        for how in ("one launch", "per layer"):
            for t in range(warm + timed):
                if t == warm:
                    torch.cuda.synchronize()
                    if how == "one launch":
                        st0 = one.stats()
                    t0 = time.perf_counter()
                if how == "one launch":
                    one.step(X[t])
                else:
                    for l, op in enumerate(each):
                        op.step(X[t][l * per:(l + 1) * per])
            torch.cuda.synchronize()
            walls[how] = (time.perf_counter() - t0) / timed * 1e6
        for l, op in enumerate(each):
            sl = slice(l * per, (l + 1) * per)
            assert torch.equal(one.slots[sl], op.slots) and torch.equal(one.miss_counts[sl], op.miss_counts)
            for s in range(ns):
                assert torch.equal(one.buffers[s][sl], op.buffers[s]), f"layer {l} stream {s}: buffers differ"
        st = one.stats()
        host_rows = (st["host_bytes"] - st0["host_bytes"]) / sum(spec.row_bytes) / timed
        row = {"strategy": name, "layers": layers, "requests_per_layer": per, "topk": spec.topk,
               "slots": spec.slots, "n_q": spec.n_q,
               "one_launch_us_per_step": round(walls["one launch"], 1),
               "per_layer_us_per_step": round(walls["per layer"], 1),
               "per_layer_over_one_launch": round(walls["per layer"] / walls["one launch"], 3),
               "host_rows_per_step": round(host_rows, 1),
               "identical": True}
        results.append(row)
        print(json.dumps(row), flush=True)
        one.close()
        for op in each:
            op.close()
    for reg in regions:
        reg.free()
    with open(out_path, "w") as f:
        json.dump(results, f, indent=1)


def _oracle_us_per_step(spec, X, N_host, host_ptrs, warm, timed):
    """The CPU oracle (match + Stage Two copy into host images of the buffers)
    on the same warm + timed steps from a cold start: µs per timed step and
    the threads it used."""
    import oracle as ORC
    _native_oracle()
    threads = ORC.default_threads()
    o = ORC.Oracle(spec.batch, spec.topk, spec.n_q, spec.slots, nthreads=threads)
    images = [np.zeros((spec.batch, spec.slots, rb), dtype=np.uint8) for rb in spec.row_bytes]
    bptr = [images[s][r].ctypes.data for s in range(len(spec.row_bytes)) for r in range(spec.batch)]
    spent = 0.0
    for t in range(warm + timed):
        N = N_host[t] if spec.speculative else None
        t0 = time.perf_counter()
        o.step(X[t], N, host=host_ptrs, buf=bptr, row_bytes=list(spec.row_bytes))
        if t >= warm:
            spent += time.perf_counter() - t0
    return spent / timed * 1e6, threads


def matching_sweep(out_path):
    """Stage One latency (matching kernel only, Stage Two off), median over 32
    timed steps after 8 warm-up steps, uniform retention 0.9, one query token:
    (a) hash vs dual-pointer at S = K = N; (b) hash, S = 4096, K = 512..4096;
    (c) hash, K = 512, S = 512..8192.  Batch 1 (one request, one workgroup)
    and batch 64."""
    import dataclasses
    import torch
    import workload as W
    from paper_2609_37538_amd import avsg as A
    dev = torch.device("cuda:0")
    ctx, rb, warm, timed = 65536, 16, 8, 32
    host = A.HostRegion(64 * ctx * rb)
    ptrs = [host.ptr + r * ctx * rb for r in range(64)]
    points = []
    for n in (256, 512, 1024, 2048):
        points += [("a", "hash", n, n), ("a", "dualptr", n, n)]
    for k in (512, 1024, 2048, 4096):
        points.append(("b", "hash", 4096, k))
    for sl in (512, 1024, 2048, 4096, 8192):
        points.append(("c", "hash", sl, 512))
    results = []
    for B in (1, 64):
        for panel, method, S, K in points:
            spec = W.custom_spec(name="match_sweep", cfg_id=11, batch=B, topk=K, slots=S, n_q=1,
                                 steps=warm + timed, ctx=ctx, retention=0.9)
            mm = A.AVSG_MATCH_DUALPTR if method == "dualptr" else A.AVSG_MATCH_HASH
            match_ms, _, d, _ = _timed_run(spec, dict(row_bytes=(rb,), match_mode=mm,
                                                      gather_mode=A.AVSG_GATHER_NONE),
                                           warm, timed, ptrs[:B], dev)
            row = {"panel": panel, "method": method, "batch": B, "S": S, "K": K,
                   "match_us_median": round(float(np.median(match_ms)) * 1e3, 2),
                   "hit_rate": round(d["hits"] / max(1, d["lookups"]), 4)}
            results.append(row)
            print(json.dumps(row), flush=True)
    host.free()
    with open(out_path, "w") as f:
        json.dump(results, f, indent=1)


def lifetime_sweep(out_path):
    """Hit rate and Stage One / Stage Two time versus the maximum lifetime L
    on a workload with reuse beyond adjacent steps: 16 requests, K = 2048,
    S = 8192, one query token, a 512-position recency window plus 1,536
    Zipf(1.1) hot positions kept step to step with p = 0.8 (16 warm-up
    steps, 48 timed).  The adjacent-step reuse of the selections is reported
    for reference."""
    import torch
    import workload as W
    from paper_2609_37538_amd import avsg as A
    dev = torch.device("cuda:0")
    B, K, S, ctx, warm, timed = 16, 2048, 8192, 1 << 20, 16, 48
    spec = W.custom_spec(name="lifetime_sweep", cfg_id=12, batch=B, topk=K, slots=S, n_q=1,
                         steps=warm + timed, ctx=ctx, mode="zipf_window", retention=0.8)
    wl = W.Workload(spec)
    X = wl.all_steps(warm + timed)
    adj = np.mean([len(np.intersect1d(X[t, r, 0], X[t - 1, r, 0])) / K
                   for t in range(warm, warm + timed) for r in range(B)])
    host = A.HostRegion(B * ctx * W.KV_ROW_BYTES)
    W.fill_host(wl, 0, host.ptr)
    ptrs = [host.ptr + r * ctx * W.KV_ROW_BYTES for r in range(B)]
    results = []
    for L in (1, 2, 4, 8, 16, 32):
        match_ms, gather_ms, d, _ = _timed_run(spec, dict(row_bytes=(W.KV_ROW_BYTES,), max_life=L),
                                               warm, timed, ptrs, dev, verified=True)
        row = {"L": L, "hit_rate": round(d["hits"] / max(1, d["lookups"]), 4),
               "adjacent_step_reuse": round(float(adj), 4),
               "match_us_median": round(float(np.median(match_ms)) * 1e3, 2),
               "gather_us_median": round(float(np.median(gather_ms)) * 1e3, 2),
               "lost_installs_per_step": round((d["lost_exhausted"] + d["lost_collision"]) / timed, 1)}
        results.append(row)
        print(json.dumps(row), flush=True)
    host.free()
    with open(out_path, "w") as f:
        json.dump(results, f, indent=1)


class _Hip:
    """The few HIP runtime calls a process without torch needs to own device
    memory (the library already loaded the runtime; same soname)."""

    def __init__(self):
        import ctypes
        self.ct = ctypes
        self.lib = ctypes.CDLL("libamdhip64.so.7")
        P, sz = ctypes.c_void_p, ctypes.c_size_t
        self.lib.hipMalloc.argtypes = [ctypes.POINTER(P), sz]
        self.lib.hipFree.argtypes = [P]
        self.lib.hipMemcpy.argtypes = [P, P, sz, ctypes.c_int]
        self.lib.hipSetDevice.argtypes = [ctypes.c_int]
        self.lib.hipStreamCreate.argtypes = [ctypes.POINTER(P)]
        self.lib.hipStreamSynchronize.argtypes = [P]
        self._check(self.lib.hipSetDevice(0), "hipSetDevice")
        self.blocks = []

    def stream(self):
        s = self.ct.c_void_p()
        self._check(self.lib.hipStreamCreate(self.ct.byref(s)), "hipStreamCreate")
        return s.value

    def _check(self, rc, what):
        if rc != 0:
            raise RuntimeError(f"{what} failed ({rc})")

    def alloc(self, nbytes):
        p = self.ct.c_void_p()
        self._check(self.lib.hipMalloc(self.ct.byref(p), max(256, int(nbytes))), "hipMalloc")
        self.blocks.append(p.value)
        return p.value

    def upload(self, dst, arr):
        self._check(self.lib.hipMemcpy(dst, arr.ctypes.data, arr.nbytes, 1), "hipMemcpy")

    def download(self, arr, src):
        self._check(self.lib.hipMemcpy(arr.ctypes.data, src, arr.nbytes, 2), "hipMemcpy")

    def sync(self):
        self._check(self.lib.hipDeviceSynchronize(), "hipDeviceSynchronize")

    def free_all(self):
        for p in self.blocks:
            self.lib.hipFree(p)
        self.blocks = []


def copy_engine_bench(out_path, names=("tiny", "batch16", "batch64_mtp2", "imbalance", "stress"),
                      warm=4, timed=16):
    """The copy-engine transfer (miss list read back, copies issued by the host)
    in a process that never loads torch: the system HIP runtime then serves
    the process and its batched copy call (one call per step for every missed
    row) is available, which the runtime PyTorch ships lacks.  Device memory
    comes from hipMalloc.  Per workload: runtime copy calls per step, Stage
    Two time (HIP events) and wall time per step, host GB/s."""
    import workload as W
    from paper_2609_37538_amd import avsg as A
    assert "torch" not in sys.modules
    A.load(share_torch_runtime=False)
    hip = _Hip()
    results = []
    for name in names:
        spec = W.get_spec(name)
        wl = W.Workload(spec)
        T = warm + timed
        B, K, nq, S = spec.batch, spec.topk, spec.n_q, spec.slots
        regions, host_ptrs = [], []
        offs = wl.request_row_offsets()
        for st, rb in enumerate(spec.row_bytes):
            reg = A.HostRegion(wl.host_rows_total() * rb)
            W.fill_host(wl, st, reg.ptr)
            regions.append(reg)
            host_ptrs += [reg.ptr + int(offs[r]) * rb for r in range(B)]
        cfg = A.make_config(B, K, nq, S, row_bytes=spec.row_bytes, gather_mode=A.AVSG_GATHER_SDMA)
        ws_bytes = A.avsg_workspace_bytes(cfg)
        ws = hip.alloc(ws_bytes)
        bufs = []
        for rb in spec.row_bytes:
            base = hip.alloc(B * S * rb)
            bufs += [base + r * S * rb for r in range(B)]
        X = np.ascontiguousarray(wl.all_steps(T), dtype=np.int32)
        Xd = hip.alloc(X.nbytes)
        hip.upload(Xd, X)
        Nd = None
        if spec.speculative:
            N = np.ascontiguousarray(np.stack([wl.verified_len(t) for t in range(T)]), dtype=np.int64)
            Nd = hip.alloc(N.nbytes)
            hip.upload(Nd, N)
        slots = hip.alloc(B * nq * K * 4)
        counts = hip.alloc(B * nq * 4)
        stream = hip.stream()       # the batched call refuses the legacy default stream
        h = A.avsg_create(cfg, host_ptrs, wl.ctx, ws, ws_bytes, bufs, stream)
        per_step = B * nq * K * 4
        try:
            for t in range(warm):
                A.avsg_step(h, Xd + t * per_step, Nd + t * B * 8 if Nd else None, slots, counts, stream)
            hip.sync()
            before = A.avsg_stats(h)
            A.avsg_set_timing(h, True)
            t0 = time.perf_counter()
            for t in range(warm, T):
                A.avsg_step(h, Xd + t * per_step, Nd + t * B * 8 if Nd else None, slots, counts, stream)
            hip.sync()
            wall = time.perf_counter() - t0
            _, gather_ms, _ = A.avsg_timing(h, timed)
            after = A.avsg_stats(h)
        finally:
            A.avsg_destroy(h)
        moved = after["host_bytes"] - before["host_bytes"]
        gsec = float(np.sum(gather_ms)) * 1e-3
        row = {"workload": name, "batch": B, "n_q": nq, "steps_timed": timed,
               "copy_calls_per_step": round((after["copy_calls"] - before["copy_calls"]) / timed, 1),
               "rows_per_step": round((after["misses"] - before["misses"]) * len(spec.row_bytes) / timed, 1),
               "gather_us_median": round(float(np.median(gather_ms)) * 1e3, 2),
               "wall_us_per_step": round(wall / timed * 1e6, 2),
               "host_gbps": round(moved / gsec / 1e9, 3) if gsec > 0 else 0.0}
        results.append(row)
        print(json.dumps(row), flush=True)
        hip.free_all()
        for reg in regions:
            reg.free()
    with open(out_path, "w") as f:
        json.dump(results, f, indent=1)


def config_table(out_path):
    """Every workload (tiny, batch16, batch64_mtp2, imbalance, stress) under the
    balanced (S3), request-level (S1), position-level (S2), copy-engine,
    pipelined, resident-reuse and early-fetch Stage Two, plus the dual-pointer matching
    ablation (S = K) on the single-token workloads: 16 warm-up steps from a
    cold start, then 64 timed steps; medians and sums from HIP events on the
    step stream, wall time between two synchronizations around the timed
    steps (with the events).  gather_gbps = bytes read over the host link /
    Stage Two time, also as fractions of the measured hipMemcpy H2D peak and
    of PCIe Gen5 x16.  Each workload also times the CPU oracle on the same
    steps."""
    import dataclasses
    import torch
    import workload as W
    from paper_2609_37538_amd import avsg as A
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cus = A.avsg_device_cus()
    warm, timed = 16, 64
    probe = A.HostRegion(512 << 20)
    tmp = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    peak = A.avsg_h2d_peak(probe.ptr, tmp.data_ptr(), 512 << 20, 20,
                           torch.cuda.current_stream(dev).cuda_stream)
    del tmp
    probe.free()
    print(json.dumps({"hipmemcpy_h2d_peak_gbps": round(peak, 3)}), flush=True)
    strategies = [("S3 balanced", A.AVSG_MATCH_HASH, A.AVSG_GATHER_BALANCED),
                  ("S1 request", A.AVSG_MATCH_HASH, A.AVSG_GATHER_REQUEST),
                  ("S2 position", A.AVSG_MATCH_HASH, A.AVSG_GATHER_POSITION),
                  ("copy engines", A.AVSG_MATCH_HASH, A.AVSG_GATHER_SDMA),
                  ("pipelined", A.AVSG_MATCH_HASH, A.AVSG_GATHER_PIPELINED),
                  ("resident reuse", A.AVSG_MATCH_HASH, A.AVSG_GATHER_RESIDENT),
                  ("early fetch", A.AVSG_MATCH_HASH, A.AVSG_GATHER_EARLY),
                  ("dual-pointer + S3", A.AVSG_MATCH_DUALPTR, A.AVSG_GATHER_BALANCED)]
    results = []
    for name in ("tiny", "batch16", "batch64_mtp2", "imbalance", "stress"):
        spec = W.get_spec(name)
        wl = W.Workload(spec)
        offs = wl.request_row_offsets()
        regions, ptrs = [], []
        for st, rb in enumerate(spec.row_bytes):
            reg = A.HostRegion(wl.host_rows_total() * rb)
            W.fill_host(wl, st, reg.ptr)
            regions.append(reg)
            ptrs += [reg.ptr + int(offs[r]) * rb for r in range(spec.batch)]
        for label, mm, gm in strategies:
            run_spec = spec
            if mm == A.AVSG_MATCH_DUALPTR:
                if spec.n_q != 1:
                    continue
                run_spec = dataclasses.replace(spec, slots=spec.topk)
            if gm == A.AVSG_GATHER_PIPELINED and spec.batch > cus:
                continue
            match_ms, gather_ms, d, wall = _timed_run(
                run_spec, dict(row_bytes=spec.row_bytes, match_mode=mm, gather_mode=gm),
                warm, timed, ptrs, dev, verified=spec.speculative)
            if gm == A.AVSG_GATHER_PIPELINED:
                gather_ms, match_ms = match_ms, None
            if gm == A.AVSG_GATHER_EARLY:
                # the list kernel, then matching beside the early copies, then
                # the finishing kernel: all of it is Stage Two's launches
                gather_ms, match_ms = gather_ms + match_ms, None
            moved = d["host_bytes"]
            gsec = float(np.sum(gather_ms)) * 1e-3
            row = {"workload": name, "strategy": label, "batch": spec.batch, "topk": spec.topk,
                   "slots": run_spec.slots, "n_q": spec.n_q,
                   "hit_rate": round(d["hits"] / max(1, d["lookups"]), 4),
                   "misses_per_step": round(d["misses"] / timed, 1),
                   "host_rows_per_step": round(d["host_bytes"] / sum(spec.row_bytes) / timed, 1),
                   "match_us_median": (round(float(np.median(match_ms)) * 1e3, 2)
                                       if match_ms is not None else None),
                   "gather_us_median": round(float(np.median(gather_ms)) * 1e3, 2),
                   "kernel_us_per_step": round((gsec + (float(np.sum(match_ms)) * 1e-3
                                                        if match_ms is not None else 0.0))
                                               / timed * 1e6, 2),
                   "wall_us_per_step": round(wall / timed * 1e6, 2),
                   "gather_gbps": round(moved / gsec / 1e9, 3) if gsec > 0 else 0.0,
                   "frac_of_hipmemcpy_peak": round(moved / gsec / 1e9 / peak, 4) if gsec > 0 else 0.0,
                   "frac_of_pcie_gen5_x16": (round(moved / gsec / 1e9 / PCIE_GEN5_X16_GBPS, 4)
                                             if gsec > 0 else 0.0),
                   "lost_installs_per_step": round((d["lost_exhausted"] + d["lost_collision"]) / timed, 1)}
            results.append(row)
            print(json.dumps(row), flush=True)
        wl_c = W.Workload(spec)
        X_c = wl_c.all_steps(warm + timed)
        N_c = np.stack([wl_c.verified_len(t) for t in range(warm + timed)])
        us, threads = _oracle_us_per_step(spec, X_c, N_c, ptrs, warm, timed)
        row = {"workload": name, "strategy": "CPU oracle", "batch": spec.batch, "topk": spec.topk,
               "slots": spec.slots, "n_q": spec.n_q, "wall_us_per_step": round(us, 1), "cores": threads}
        results.append(row)
        print(json.dumps(row), flush=True)
        for reg in regions:
            reg.free()
    with open(out_path, "w") as f:
        json.dump(results, f, indent=1)


# sources that decide the profiled kernel's traffic: the gather code and the
# matching code that plans which rows it reads
GATHER_SOURCES = ("paper_2609_37538_amd/csrc/gather.hip", "paper_2609_37538_amd/csrc/gather_body.h",
                  "paper_2609_37538_amd/csrc/match_body.h", "paper_2609_37538_amd/csrc/avsg_internal.h")
TRAFFIC_SUMMARY = "profiles/gather_resident_traffic_batch64_mtp2.md"
TRAFFIC_SUMMARY_S3 = "profiles/gather_balanced_traffic_batch64_mtp2.md"


def measured_traffic(args, gather_name):
    """HBM + host-link bytes per gather launch from the committed rocprofv3
    counter summary (FETCH_SIZE x 2.0 + WRITE_SIZE x 1.0, copy-calibrated), or
    None when this run is not the profiled workload and transfer or the gather
    source has changed since the counters were taken.  The counters were
    taken over the steady-state launches of one run of the workload; a step's
    traffic changes little from step to step (the summary names its sample)."""
    if (args.config, args.workers, gather_name, args.match) != ("batch64_mtp2", 0, "resident", "hash"):
        return None
    return _traffic_block(TRAFFIC_SUMMARY)


def _traffic_block(summary):
    """The JSON block of a committed counter summary, or None when the gather
    and matching code has changed since it was taken."""
    import re
    path = os.path.join(ROOT, summary)
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
    if not m:
        return None
    block = json.loads(m.group(1))
    if gather_code_hash() != block.get("source_sha256_16"):
        return None
    return block


def gather_code_hash(root=None):
    """First 16 hex digits of the SHA-256 of the code of GATHER_SOURCES with
    comments and whitespace removed (a comment edit keeps the counters valid;
    any code change invalidates them)."""
    import hashlib
    import re
    h = hashlib.sha256()
    for p in GATHER_SOURCES:
        text = open(os.path.join(root or ROOT, p), encoding="utf-8").read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def cpu_baseline(spec, wl, X_host, N_host, host_ptrs, args, gather_mode):
    """Time the oracle (match + Stage Two copy into host images of the buffers)
    on the warmup+timed steps of the same workload, from the same cold start;
    report µs per timed step."""
    import oracle as ORC
    build = _native_oracle()
    threads = ORC.default_threads()
    o = ORC.Oracle(spec.batch, spec.topk, spec.n_q, spec.slots, nthreads=threads)
    images = [np.zeros((spec.batch, spec.slots, rb), dtype=np.uint8) for rb in spec.row_bytes]
    bptr = [images[s][r].ctypes.data for s in range(len(spec.row_bytes)) for r in range(spec.batch)]
    T = X_host.shape[0]
    n_run = T if args.cpu_sample_steps <= 0 else min(T, args.cpu_sample_steps)
    first_timed = min(args.warmup, n_run - 1)
    timed = 0.0
    n_timed = 0
    gather = gather_mode != 3
    for t in range(n_run):
        N = N_host[t] if spec.speculative else None
        t0 = time.perf_counter()
        if gather:
            o.step(X_host[t], N, host=host_ptrs, buf=bptr, row_bytes=list(spec.row_bytes))
        else:
            o.step(X_host[t], N)
        dt = time.perf_counter() - t0
        if t >= first_timed:
            timed += dt
            n_timed += 1
    # the same oracle on one thread, over a shorter run (cold start + warmup + 8 timed steps)
    o1 = ORC.Oracle(spec.batch, spec.topk, spec.n_q, spec.slots, nthreads=1)
    n1 = min(n_run, first_timed + 8)
    t1 = 0.0
    for t in range(n1):
        N = N_host[t] if spec.speculative else None
        t0 = time.perf_counter()
        if gather:
            o1.step(X_host[t], N, host=host_ptrs, buf=bptr, row_bytes=list(spec.row_bytes))
        else:
            o1.step(X_host[t], N)
        if t >= first_timed:
            t1 += time.perf_counter() - t0
    return {
        "value": round(timed / max(1, n_timed) * 1e6, 1),
        "unit": "us/step",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{spec.name} steps {first_timed}..{n_run - 1} ({n_timed} steps) after a cold start "
                  f"at step 0, match + Stage Two copy into host images, {threads} OpenMP threads",
        "single_thread_us_per_step": round(t1 / max(1, n1 - first_timed) * 1e6, 1),
        "single_thread_sample": f"steps {first_timed}..{n1 - 1} of the same run",
        "cpu_model": _cpu_model(),
        "affinity_cpus": ORC.affinity_cpus(),
        "thread_cap": ORC.thread_cap(),
        "build": build,
    }


_NATIVE = None


def _native_oracle():
    """Build the oracle with -O3 -march=native on this host (into a temporary
    directory) and make it the one the oracle package loads; returns the
    build's description.  Falls back to the in-tree -O3 build when gcc is
    unavailable.  Must run before the oracle is first used in the process."""
    global _NATIVE
    if _NATIVE is not None:
        return _NATIVE
    import tempfile
    import oracle as ORC
    if ORC._lib is not None:
        _NATIVE = "gcc -O3 (in-tree build, already loaded)"
        return _NATIVE
    try:
        out = os.path.join(tempfile.mkdtemp(prefix="avsg_oracle_"), "liboracle_avsg_native.so")
        ORC.build(force=True, native=True, out=out)
        os.environ["AVSG_ORACLE_LIB"] = out
        _NATIVE = "gcc -O3 -march=native -fopenmp, built on this host"
    except (OSError, subprocess.CalledProcessError):
        _NATIVE = "gcc -O3 -fopenmp (in-tree build)"
    return _NATIVE


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
