#!/usr/bin/env python3
"""Benchmark of one CP rank's prefill-attention hot path on one MI355X.

A step is one pass of the whole path for rank 0 of the workload:
  1. the zigzag shard plan (host, cp_shard_plan);
  2. partial attention of the rank's rows -- one cp_attn_partial launch:
     by default (--mode allgather) against every key the rank's rows see in
     the all-gathered KV (and the paged prefix, if any), one descriptor whose
     output rows are stored at their places in the original sequence order
     (CP_OUT_SEQUENCE: the restore done by the attention's own stores);
     with --mode passkv against each of the C ranks' KV shards (and the
     prefix) separately, C (+1) descriptors in local row order;
  3. --mode passkv only: cp_attn_merge with the plan, the exact LSE merge of
     the partials, writing each row back to its place in sequence order.
Inputs are resident in HBM before the timed region starts.  In the
all-gather view the merge object reports a separate leg: C (+1) partials of
the same rows (seeded values, every LSE finite, so every partial is read)
merged and restored.

value  = 4 * D * Hq * visible_pairs / step time  (TFLOP/s; the two MFMA
         contractions per visible query-key pair, no credit for masked work).
roofline = the partial-attention kernel: the same FLOPs / its average launch
         duration from HIP events on its stream, against 2.5 PFLOP/s dense bf16.
cpu_baseline = the fp64 oracle on a bounded sample of the same rows.

Usage: python bench.py [--steps K] [--warmup W] [--workload NAME] [--mode passkv|allgather]
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

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
NOMINAL_CLOCK_GHZ = 2.4        # the clock the bf16 peak is quoted at
METRIC = "CP-shard causal prefill attention TFLOP/s + % bf16 MFMA peak; merge GB/s"
DEFAULT_WORKLOAD = "llama3_8b_32k_c4"


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--rank", type=int, default=0)
    ap.add_argument("--mode", choices=["passkv", "allgather"], default="allgather")
    ap.add_argument("--hetero", action="store_true",
                    help="also time the heterogeneous batch (64 requests, one varlen launch); off by default so "
                         "that a kernel trace of the default run holds only the workload's attention launches")
    ap.add_argument("--c-rule", choices=["cost", "length", "both"], default="both",
                    help="per-request CP degree of the heterogeneous batch: the placement cost over the "
                         "calibrated prefill-time model, the fixed length rule, or both (each timed)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="wall-clock budget of the CPU oracle sample (0 disables it)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="before timing, copy this many MiB once with repartition_kernel (plain "
                         "16-byte loads and stores), so that a counter profile of the run can scale "
                         "FETCH_SIZE/WRITE_SIZE by a known size")
    return ap.parse_args()


def profiled_figures(workload, mode="allgather"):
    """Figures of the committed counter profile of this workload's launch in
    this mode (HBM bytes per attention launch, and where recorded the clock
    and MFMA-busy fraction), if the kernel and planner sources are still the
    ones that were profiled (the plan decides which items are cut, and the
    pieces' partials are traffic too)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}_{mode}.txt")
    src = os.path.join(ROOT, "paper_2609_04774_amd", "csrc", "attn_partial.hip")
    planner = os.path.join(ROOT, "paper_2609_04774_amd", "csrc", "cp_attn.cpp")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        line = line.strip()
        if line and not line.startswith("#") and "=" in line:
            key, val = line.split("=", 1)
            kv[key] = val
    with open(src, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()
    with open(planner, "rb") as f:
        planner_sha = hashlib.sha256(f.read()).hexdigest()
    if kv.get("kernel_source_sha256") != sha or kv.get("planner_source_sha256") != planner_sha:
        return None
    if kv.get("mode") != mode:
        return None
    out = {"traffic": int(kv["fetch_bytes"]) + int(kv["write_bytes"])}
    if "clock_ghz" in kv and "mfma_busy" in kv:
        out["clock_ghz"] = float(kv["clock_ghz"])
        out["mfma_busy"] = float(kv["mfma_busy"])
    return out


def measured_traffic(workload, mode="allgather"):
    """HBM bytes per attention launch from the committed counter profile."""
    f = profiled_figures(workload, mode)
    return None if f is None else f["traffic"]


CALIBRATION = os.path.join(ROOT, "profiles", "calibration_attention_llama3_8b.json")


def heterogeneous_batch(args, gen, dev, stream, reps=5):
    """The varlen launch: 64 requests of lognormal length (median 2048, clipped
    to 256..131072), 19 of them with a cached prefix in one shared paged pool
    -- every (request, rank) shard's partial over all its visible keys in one
    cp_attn_partial launch.  Each request's CP degree comes from the placement
    cost (PreferDegree over the calibrated prefill-time model) and, for
    comparison, from the fixed length rule; the same seeded data is run under
    each rule chosen by --c-rule."""
    import torch

    import synth
    from paper_2609_04774_amd import cpattn as cp
    from paper_2609_04774_amd import placement as pl

    Hq, Hkv, D, B = 32, 8, 128, synth.BLOCK_TOKENS
    reqs = synth.hetero_requests()
    model = pl.model_from_calibration(CALIBRATION)
    total_blocks = sum(P // B for _, P in reqs) + 32
    k_pool = synth.randn_bf16(gen, (total_blocks, B, Hkv, D), device="cuda")
    v_pool = synth.randn_bf16(gen, (total_blocks, B, Hkv, D), device="cuda")
    free = torch.randperm(total_blocks, generator=gen, device="cuda")
    used = 0
    data = []
    for L, P in reqs:
        R = L - P
        q_full, k, v = synth.qkv(gen, R, R, Hq, Hkv, D, device="cuda")
        table = None
        if P:
            pre = synth.paged_prefix(gen, P, Hkv, D, device="cuda",
                                     pool=(k_pool, v_pool, free[used:used + P // B]))
            used += P // B
            table = pre.block_table
        data.append((L, P, R, q_full, k, v, table))
    out = {
        "kernel": "attn_partial_kernel", "requests": len(reqs), "tokens": sum(L for L, _ in reqs),
        "prefixed": sum(1 for _, P in reqs if P),
        "degree_model": {"source": os.path.relpath(CALIBRATION, ROOT), "d0_s": model.d, "alpha_s": model.alpha,
                         "beta": pl.DEFAULT_BETA, "lambda": pl.DEFAULT_LAMBDA},
    }
    rules = ["cost", "length"] if args.c_rule == "both" else [args.c_rule]
    for rule in rules:
        degrees = pl.choose_degrees(reqs, rule, model)
        keep, descs = [], []
        pairs = 0
        for (L, P, R, q_full, k, v, table), C in zip(data, degrees):
            for r in range(C):
                plan, rows = cp.shard_plan(P, R, C, r)
                if plan.n_rows == 0:
                    continue
                q = q_full[torch.as_tensor(rows - P, device=dev)].contiguous()
                o = torch.empty((plan.n_rows, Hq, D), dtype=torch.float32, device=dev)
                lse = torch.empty((plan.n_rows, Hq), dtype=torch.float32, device=dev)
                descs.append(cp.make_desc(plan, q, k, v, o, lse, k_pool, v_pool, table, include_prefix=True))
                keep.append((q, o, lse))
                pairs += plan.visible_pairs
        ws = torch.empty(max(256, cp.workspace_size(descs, Hq, Hkv)), dtype=torch.uint8, device=dev)
        for _ in range(2):
            cp.attn_partial(descs, Hq, Hkv, ws, stream=stream)
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            cp.attn_partial(descs, Hq, Hkv, ws, stream=stream)
        b.record(stream)
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / reps
        flop = 4.0 * D * Hq * pairs
        out[rule] = {
            "C_histogram": {str(C): degrees.count(C) for C in pl.DEGREES},
            "descriptors": len(descs), "flop": flop, "ms": round(ms, 4),
            "TFLOP_s": round(flop / (ms * 1e-3) / 1e12, 2),
            "frac": round(flop / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        }
        del keep, descs, ws
    del data, k_pool, v_pool
    return out


def counter_profile(workload, args, rank, frac):
    """The committed counter profile's clock and MFMA-busy fraction for this
    launch configuration (null when there is none for the current source),
    and this run's fraction of peak re-based to that sustained clock: the
    peak the matrix cores can reach at the clock the chip holds under this
    load (2.5 PFLOP/s x clock / 2.4 GHz)."""
    if rank != 0:
        return None
    f = profiled_figures(workload, args.mode)
    if f is None or "clock_ghz" not in f:
        return None
    return {"clock_ghz": f["clock_ghz"], "mfma_busy": f["mfma_busy"],
            "frac_at_profiled_clock": round(frac * NOMINAL_CLOCK_GHZ / f["clock_ghz"], 4),
            "source": f"profiles/traffic_{workload}_{args.mode}.txt "
                      "(rocprofv3 GRBM_GUI_ACTIVE, SQ_VALU_MFMA_BUSY_CYCLES)"}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library executes every CP rank's shard "
              "on a single MI355X and has no multi-GPU path (--gpus must be 1).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2609_04774_amd import cpattn as cp

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    w = synth.WORKLOADS[args.workload]
    P, R, C, Hq, Hkv, D = w.P, w.R, w.C, w.Hq, w.Hkv, w.D
    rank = args.rank
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    # --- inputs, resident in HBM -------------------------------------------
    plan, rows = cp.shard_plan(P, R, C, rank)
    n_rows = plan.n_rows
    gen = synth.generator(w.seed + 100 * rank, device="cuda")
    q = synth.randn_bf16(gen, (n_rows, Hq, D), w.data_scale, device="cuda")
    k = synth.randn_bf16(gen, (R, Hkv, D), w.data_scale, device="cuda")
    v = synth.randn_bf16(gen, (R, Hkv, D), w.data_scale, device="cuda")
    prefix = synth.paged_prefix(gen, P, Hkv, D, w.data_scale, spare_blocks=64, device="cuda") if P else None
    kc = prefix.k_cache if prefix else None
    vc = prefix.v_cache if prefix else None
    bt = prefix.block_table if prefix else None

    if args.mode == "passkv":
        shard_ids = list(range(C))
        n_parts = C + (1 if P else 0)
    else:
        shard_ids = [cp.CP_KV_ALL]
        n_parts = 1
    out = torch.empty((R, Hq, D), dtype=torch.float32, device=dev)
    out_lse = torch.empty((R, Hq), dtype=torch.float32, device=dev)
    if args.mode == "passkv":
        o_parts = torch.empty((n_parts, n_rows, Hq, D), dtype=torch.float32, device=dev)
        l_parts = torch.empty((n_parts, n_rows, Hq), dtype=torch.float32, device=dev)

    def make_descs(pl):
        descs = []
        i = 0
        if args.mode == "passkv" and P:
            descs.append(cp.make_desc(pl, q, k, v, o_parts[i], l_parts[i], kc, vc, bt,
                                      include_prefix=True, kv_rank=cp.CP_KV_NONE))
            i += 1
        if args.mode == "allgather":
            return [cp.make_desc(pl, q, k, v, out, out_lse, kc, vc, bt, include_prefix=True,
                                 kv_rank=cp.CP_KV_ALL, out_order=cp.CP_OUT_SEQUENCE)]
        for s in shard_ids:
            descs.append(cp.make_desc(pl, q, k, v, o_parts[i], l_parts[i], kc, vc, bt,
                                      include_prefix=False, kv_rank=s))
            i += 1
        return descs

    ws = torch.empty(max(256, cp.workspace_size(make_descs(plan), Hq, Hkv)), dtype=torch.uint8, device=dev)
    if args.copy_calibration_mib > 0:
        # A plain copy of known size (repartition_kernel from degree 1 to degree 1:
        # every row read once and written once with ordinary 16-byte loads and
        # stores), so that a counter profile can scale FETCH_SIZE/WRITE_SIZE.
        n_cal = (args.copy_calibration_mib << 20) // (Hkv * D * 2)
        src = torch.ones((n_cal, Hkv, D), dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        cp.repartition(0, n_cal, [src], 1, 0, dst)
        torch.cuda.synchronize()
        del src, dst
    stream = torch.cuda.current_stream()
    flop = 4.0 * D * Hq * plan.visible_pairs

    ev = []

    def step(record):
        pl, _ = cp.shard_plan(P, R, C, rank, with_rows=False)
        descs = make_descs(pl)
        e0 = e1 = e2 = None
        if record:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e2 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
        cp.attn_partial(descs, Hq, Hkv, ws, stream=stream)
        if record:
            e1.record(stream)
        if args.mode == "passkv":
            cp.attn_merge([o_parts[i] for i in range(n_parts)], [l_parts[i] for i in range(n_parts)],
                          out, out_lse, restore=pl, stream=stream)
        if record:
            e2.record(stream)
            ev.append((e0, e1, e2))

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    attn_ms = sum(a.elapsed_time(b) for a, b, _ in ev) / len(ev)
    merge_ms = sum(b.elapsed_time(c) for _, b, c in ev) / len(ev)

    rows_merged = n_rows * Hq
    attn_tflops = flop / (attn_ms * 1e-3) / 1e12
    value = flop / (ms_step * 1e-3) / 1e12

    def timed(fn, reps=10):
        """GPU time per call of fn (its launches back to back).  A GPU-side
        wait is queued first, so that every repetition is enqueued before the
        GPU reaches them: for launches shorter than the binding's own host
        time the events then bracket the kernels, not the host's call rate."""
        fn()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(5_000_000)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    # --- the merge ----------------------------------------------------------
    # Algorithmic bytes: every partial's LSE, the O of each partial whose LSE
    # is finite (a partial of weight 0 is not read), the merged O and LSE.
    if args.mode == "passkv":
        n_merged = n_parts
        finite = int(torch.isfinite(l_parts).sum().item())
        merge_what = (f"the step's merge of the {n_parts} pass-KV partials with restore "
                      "(O of a partial with LSE = -inf is not read)")
    else:
        n_merged = C + (1 if P else 0)
        m_o = torch.randn((n_merged, n_rows, Hq, D), generator=gen, device=dev)
        m_l = 3.0 * torch.randn((n_merged, n_rows, Hq), generator=gen, device=dev)
        m_out = torch.empty_like(out)
        m_lse = torch.empty_like(out_lse)
        merge_ms = timed(lambda: cp.attn_merge([m_o[i] for i in range(n_merged)], [m_l[i] for i in range(n_merged)],
                                               m_out, m_lse, restore=plan, stream=stream))
        finite = n_merged * rows_merged
        merge_what = (f"{n_merged} partials of the rank's rows (seeded values, every LSE finite) "
                      "merged with restore, as after pass-KV partials")
        del m_o, m_l, m_out, m_lse
    merge_bytes = finite * 4 * D + n_merged * rows_merged * 4 + rows_merged * (4 * D + 4)
    merge_gbs = merge_bytes / (merge_ms * 1e-3) / 1e9

    # --- the KV-cache steps after the attention (not part of the timed step) --
    # All C ranks of the request, as one GPU per rank would each do for its own.
    rank_rows = [torch.as_tensor(cp.shard_plan(P, R, C, r)[1] - P, device=dev) for r in range(C)]
    plans = [cp.shard_plan(P, R, C, r)[0] for r in range(C)]
    k_ranks = [k[ix].contiguous() for ix in rank_rows]
    v_ranks = [v[ix].contiguous() for ix in rank_rows]
    n_req_blocks = -(-(P + R) // synth.BLOCK_TOKENS)
    wb_table = torch.randperm(n_req_blocks, generator=gen, device="cuda").to(torch.int32)
    k_store = torch.empty((n_req_blocks, synth.BLOCK_TOKENS, Hkv, D), dtype=torch.bfloat16, device=dev)
    v_store = torch.empty_like(k_store)

    def writeback():
        for r in range(C):
            cp.kv_writeback(plans[r], k_ranks[r], v_ranks[r], k_store, v_store, wb_table, stream=stream)

    wb_ms = timed(writeback)
    wb_bytes = 2 * 2 * R * Hkv * D * 2                # K and V rows, read once and written once
    dst_plans = [cp.shard_plan(P, R, 2 * C, r)[0] for r in range(2 * C)]
    dst_k = [torch.empty((pl.n_rows, Hkv, D), dtype=torch.bfloat16, device=dev) for pl in dst_plans]
    dst_v = [torch.empty_like(t) for t in dst_k]

    def reshard():
        # Every degree-2C rank's K and V rows in one launch.
        cp.repartition_all(P, R, [k_ranks, v_ranks], [dst_k, dst_v], stream=stream)

    rp_ms = timed(reshard)
    rp_bytes = 2 * 2 * R * Hkv * D * 2                # K and V rows, read once and written once
    del k_ranks, v_ranks, dst_k, dst_v, k_store, v_store

    # The paged gather on its own: a 48K-token cached prefix (the prefix-hit
    # workload's, 3072 blocks of 16 under a permuted table) read back out of
    # the paged cache into contiguous K and V rows, one launch.
    P_g = synth.WORKLOADS["prefix_hit_64k_c2"].P
    pre_g = synth.paged_prefix(gen, P_g, Hkv, D, 1.0, spare_blocks=64, device="cuda")
    k_g = torch.empty((P_g, Hkv, D), dtype=torch.bfloat16, device=dev)
    v_g = torch.empty_like(k_g)
    ga_ms = timed(lambda: cp.kv_gather(pre_g.k_cache, pre_g.v_cache, pre_g.block_table, 0, k_g, v_g,
                                       stream=stream))
    ga_bytes = 2 * 2 * P_g * Hkv * D * 2             # K and V rows, read once and written once
    del pre_g, k_g, v_g

    hetero = heterogeneous_batch(args, gen, dev, stream) if args.hetero else None

    # --- CPU oracle on a bounded sample of the same rows ----------------------
    cpu = None
    parity = None
    if args.cpu_seconds > 0:
        cpu, parity = cpu_baseline(args, w, plan, rows, q, k, v, prefix, out, out_lse, flop)

    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name, "L": w.L, "P": P, "R": R, "C": C, "rank": rank, "Hq": Hq,
            "Hkv": Hkv, "D": D, "rows": n_rows, "visible_pairs_per_head": plan.visible_pairs,
            "flop_per_step": flop, "mode": ("pass-KV partials + LSE merge + restore" if args.mode == "passkv"
                                            else "all-gathered KV partial stored in sequence order"),
            "partials": n_parts,
        },
        "pct_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "roofline": {
            "kernel": "attn_partial_kernel",
            "bound": "mfma",
            "achieved": round(attn_tflops, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": measured_traffic(w.name, args.mode) if rank == 0 else None,
            "launch_ms": round(attn_ms, 4),
            "profiled": counter_profile(w.name, args, rank, attn_tflops / PEAK_BF16_TFLOPS),
        },
        "merge": {
            "kernel": "lse_merge_kernel", "bound": "hbm", "ms": round(merge_ms, 4),
            "bytes": merge_bytes, "GB_s": round(merge_gbs, 1),
            "frac": round(merge_gbs / PEAK_HBM_GBS, 4), "partials": n_merged, "what": merge_what,
        },
        "kv_writeback": {
            "kernel": "kv_writeback_kernel", "bound": "hbm", "ms": round(wb_ms, 4), "bytes": wb_bytes,
            "GB_s": round(wb_bytes / (wb_ms * 1e-3) / 1e9, 1),
            "frac": round(wb_bytes / (wb_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "what": "every rank's new K and V rows into the block-16 paged cache (C launches)",
        },
        "paged_gather": {
            "kernel": "kv_gather_kernel", "bound": "hbm", "ms": round(ga_ms, 4), "bytes": ga_bytes,
            "GB_s": round(ga_bytes / (ga_ms * 1e-3) / 1e9, 1),
            "frac": round(ga_bytes / (ga_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "what": "a 49152-token paged prefix (permuted block-16 table) read back into contiguous K and V rows",
        },
        "heterogeneous_batch": hetero,
        "repartition": {
            "kernel": "repartition_all_kernel", "bound": "hbm", "ms": round(rp_ms, 4), "bytes": rp_bytes,
            "GB_s": round(rp_bytes / (rp_ms * 1e-3) / 1e9, 1),
            "frac": round(rp_bytes / (rp_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "what": "the request's K and V rows re-sharded from degree C to degree 2C, every destination "
                    "rank in one launch (cp_repartition_all)",
        },
        "cpu_baseline": cpu,
        "parity_sample": parity,
    }
    print(json.dumps(line), flush=True)


def cpu_baseline(args, w, plan, rows, q, k, v, prefix, out, out_lse, flop_total):
    """Time the oracle (as it stands) on seeded rows of the same shard, and
    compare those rows with the GPU's merged output on the way."""
    import numpy as np
    import torch

    from oracle import attention as oatt

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    cores_available = len(os.sched_getaffinity(0))
    P, R, Hq, D = w.P, w.R, w.Hq, w.D
    kk = k.cpu().double().numpy()
    vv = v.cpu().double().numpy()
    if prefix is not None:
        bt = prefix.block_table.cpu().numpy().astype(np.int64)
        kc = prefix.k_cache.cpu().double().numpy()
        vc = prefix.v_cache.cpu().double().numpy()
    else:
        bt = kc = vc = None
    rng = np.random.default_rng(w.seed)
    order = rng.permutation(plan.n_rows)
    # Always include both chunks' first and last rows.
    c0 = plan.chunk[0].q_len
    firsts = [0, max(0, c0 - 1), c0, plan.n_rows - 1]
    order = list(dict.fromkeys([i for i in firsts if 0 <= i < plan.n_rows] + list(order)))
    done_rows, pairs, err_o, err_l = [], 0, 0.0, 0.0
    t0 = time.perf_counter()
    batch = 2
    while order and time.perf_counter() - t0 < args.cpu_seconds:
        take, order = order[:batch], order[batch:]
        idx = np.array(take, dtype=np.int64)
        pos = rows[idx]
        qq = q[torch.as_tensor(idx, device=q.device)].cpu().double().numpy()
        O, L = oatt.rank_partial(qq, pos, P, kk, vv, kc, vc, bt)
        pairs += int(np.sum(pos + 1))
        done_rows.extend(take)
        g_o = out[torch.as_tensor(pos - P, device=out.device)].cpu().double().numpy()
        g_l = out_lse[torch.as_tensor(pos - P, device=out.device)].cpu().double().numpy()
        err_o = max(err_o, float(np.max(np.abs(g_o - O))))
        err_l = max(err_l, float(np.max(np.abs(g_l - L))))
    elapsed = time.perf_counter() - t0
    flop = 4.0 * D * Hq * pairs
    cpu = {
        "value": round(flop / elapsed / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": int(threads),
        "cores_available": cores_available,
        "cpu_model": cpu_model,
        "kind": "oracle",
        "sample": f"{len(done_rows)} of {plan.n_rows} rank-{plan.rank} rows x {Hq} heads over all their "
                  f"visible keys (fp64 numpy), {elapsed:.1f} s",
        "seconds": round(elapsed, 2),
        "est_full_step_s": round(flop_total / (flop / elapsed), 1) if flop else None,
    }
    parity = {"rows": len(done_rows), "max_abs_o": err_o, "max_abs_lse": err_l,
              "ok": bool(err_o <= 1e-2 and err_l <= 1e-3)}
    return cpu, parity


if __name__ == "__main__":
    main()
