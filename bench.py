#!/usr/bin/env python3
"""Benchmark: multi-stage live migration of a request's paged KV cache on one
MI355X (Llumnix §4.2), through the llmig C ABI.

One step is one whole migration of the LLaMA-7B-shaped request: 32 layers,
32 KV heads of 128, 16-token blocks, fp16, pools of 4096 blocks with 40% of
each held by other requests; stage 1 copies the 8192 resident tokens (512
blocks), then four times decoding appends 16-64 tokens (seeded) and a stage
copies the new whole blocks, the fourth stage being final (drain + copy the
rest).  Inputs are resident in HBM before timing starts.

value = algorithmic bytes read + written by all stages / wall time per step.
The JSON line also carries the roofline of the dominant kernel (the bulk
pool-to-pool copy of stage 1), the CPU oracle's rate on a bounded sample, and
the final-stage downtime against sequence length for the LLaMA-30B
tensor-parallel-quarter shape (60 layers, 13 heads of 128; 1k/4k/16k tokens).

    python bench.py [--steps K] [--warmup W] [--gpus 1]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def recorded_traffic(kernel: str):
    """HBM bytes per launch of ``kernel`` from the committed counter summary
    (two rocprofv3 --pmc passes, calibrated against a plain copy), or None
    when the kernel source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "copy_tiles_bulk_llama7b_traffic.txt")
    src = os.path.join(ROOT, "paper_2406_03243_amd", "csrc", "llmig.hip")
    try:
        rec = json.load(open(path))
        now = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except (OSError, ValueError):
        return None
    if rec.get("kernel") != kernel or rec.get("kernel_source_sha256") != now:
        return None
    return rec["traffic_bytes_per_launch"]


def stage_bytes(blocks, shape, tile_bytes):
    """Algorithmic bytes of a stage: every tile read once and written once."""
    return 2 * blocks * shape.num_layers * 2 * tile_bytes


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="CPU oracle sample budget")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-downtime-sweep", action="store_true")
    ap.add_argument("--downtime-reps", type=int, default=7)
    ap.add_argument("--calibration-copy", action="store_true",
                    help="end with two plain 1 GiB device-to-device copies (hardware counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures migration between two block pools on one GPU; "
              "no multi-GPU configuration exists (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2406_03243_amd.build import LIBRARY
    if not os.path.exists(LIBRARY):
        import __graft_entry__
        __graft_entry__.build()
    from paper_2406_03243_amd import harness, migrate
    from paper_2406_03243_amd import workloads as wl
    from paper_2406_03243_amd.llmig import Pool

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    # ------------------------------------------------------------------ workload
    w = wl.LLAMA7B
    shape = w.shape
    log("allocating", w.name, shape)
    sk, sv = harness.alloc_layers(shape, device=dev)
    dk, dv = harness.alloc_layers(shape, device=dev)
    harness.fill_on_device(sk + sv, w.seed * 16 + wl.SRC_VALUES)
    harness.fill_on_device(dk + dv, w.seed * 16 + wl.DST_VALUES)
    src, dst = Pool(sk, sv), Pool(dk, dv)
    table, _ = wl.request_table(w.seed, shape.num_blocks, w.table_blocks, w.src_preoccupied)
    free, _ = wl.free_list(w.seed, shape.num_blocks, w.dst_preoccupied)
    counts = wl.append_counts(w.seed, w.appends, w.append_lo, w.append_hi)
    appends = []
    for k, c in enumerate(counts):
        bits = wl.values16(w.seed, wl.APPEND_VALUES, shape.num_layers * 2 * int(c) * src.slot_bytes // 2,
                           shape.dtype, sub=k)
        appends.append(torch.from_numpy(bits.view(np.uint8)).to(dev))
    initial = w.lengths[0]
    mig, dec = torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()

    def step():
        return migrate.run_scheduled(src, dst, table, free, initial, appends, mig, dec)

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    log(f"timing {args.steps} steps")
    runs = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        runs.append(step())
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    m0 = runs[0][0]
    blocks_per_step = sum(r.blocks for r in m0.stages)
    bytes_per_step = stage_bytes(blocks_per_step, shape, src.tile_bytes)
    ms_per_step = elapsed / args.steps * 1e3
    value = bytes_per_step / (elapsed / args.steps) / 1e9

    # dominant kernel: the bulk pool-to-pool copy of stage 1, launched on the
    # migration stream; its ids travel in the kernel arguments, 256 pairs per launch
    s1_blocks = m0.stages[0].blocks
    launches = math.ceil(s1_blocks / 256)
    s1_us = [m.stages[0].gpu_us for m, _ in runs]
    s1_avg_us = statistics.fmean(s1_us)
    per_launch_bytes = stage_bytes(s1_blocks, shape, src.tile_bytes) / launches
    per_launch_us = s1_avg_us / launches
    achieved = per_launch_bytes / (per_launch_us * 1e-6) / 1e9
    downtimes = [d for _, d in runs]
    kernel_name = "copy_tiles<0, 0, true, %d>" % (16 if src.tile_bytes >= 32 * 4096 else 8)

    stages = []
    for i, rec in enumerate(m0.stages):
        us = [m.stages[i].gpu_us for m, _ in runs if m.stages[i].gpu_us > 0]
        b = stage_bytes(rec.blocks, shape, src.tile_bytes)
        entry = {"tokens": [rec.from_tok, rec.to_tok], "blocks": rec.blocks, "bytes": b, "final": rec.final}
        if us:
            entry["gpu_us_median"] = round(statistics.median(us), 2)
            entry["GBps"] = round(b / (statistics.median(us) * 1e-6) / 1e9, 1)
        stages.append(entry)

    result = {
        "metric": "KV migration GB/s (fraction of HBM peak); final-stage downtime us vs seq len",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": w.name, "layers": shape.num_layers, "kv_heads": shape.kv_heads,
                   "head_dim": shape.head_dim, "block_size": shape.block_size, "elem": shape.dtype,
                   "pool_blocks": shape.num_blocks, "preoccupied": w.src_preoccupied,
                   "initial_tokens": initial, "appended": [int(c) for c in counts],
                   "bytes_per_step": bytes_per_step},
        "fraction_of_hbm_peak": round(value / HBM_PEAK_GBS, 4),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": recorded_traffic(kernel_name),
                     "kernel": kernel_name,
                     "launches_per_stage": launches, "bytes_per_launch": int(per_launch_bytes),
                     "avg_launch_us": round(per_launch_us, 2)},
        "stages": stages,
        "final_stage_downtime_us": {"median": round(statistics.median(downtimes), 1),
                                    "min": round(min(downtimes), 1), "max": round(max(downtimes), 1)},
    }

    # ------------------------------------------------------------------ CPU oracle baseline
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(src, m0.stages[0], shape, args.cpu_seconds)

    if args.calibration_copy:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        a.fill_(1)
        for _ in range(2):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    del appends
    src.close()
    dst.close()
    del sk, sv, dk, dv, src, dst
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    # ------------------------------------------------------------------ downtime vs length
    if not args.no_downtime_sweep:
        result["downtime_vs_len"] = downtime_sweep(args.downtime_reps)

    print(json.dumps(result), flush=True)


def cpu_baseline(src, stage1, shape, seconds):
    """The oracle's per-tile copy on host snapshots of a sample of stage 1's
    blocks, single-threaded, repeated for about ``seconds``."""
    import numpy as np

    import oracle
    from oracle import HostPool
    from paper_2406_03243_amd import harness

    n = 64
    ms, md = stage1.map_src[:n], stage1.map_dst[:n]
    hs = HostPool(harness.snapshot_blocks(src.k, ms), harness.snapshot_blocks(src.v, ms),
                  src.block_size, src.slot_bytes)
    hd = HostPool.zeros(shape.num_layers, n, src.block_size, src.slot_bytes)
    ids = np.arange(n, dtype=np.int32)
    orc = oracle.default()
    orc.copy(hs, hd, ids, ids)           # warm the pages
    reps, t0 = 0, time.perf_counter()
    while True:
        orc.copy(hs, hd, ids, ids)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    moved = reps * 2 * n * shape.num_layers * 2 * src.tile_bytes
    return {"value": round(moved / el / 1e9, 2), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{n} of the {stage1.blocks} stage-1 block pairs (all {shape.num_layers} layers, "
                      f"K and V, {n * shape.num_layers * 2} tiles of {src.tile_bytes} B) copied {reps} times "
                      f"from host snapshots, {el:.1f} s, one thread"}


def downtime_sweep(reps):
    import numpy as np
    import torch

    from paper_2406_03243_amd import harness, migrate
    from paper_2406_03243_amd import workloads as wl
    from paper_2406_03243_amd.llmig import Pool

    w = wl.LLAMA30B_TP4
    shape = w.shape
    log("allocating", w.name, shape)
    sk, sv = harness.alloc_layers(shape)
    dk, dv = harness.alloc_layers(shape)
    harness.fill_on_device(sk + sv, w.seed * 16 + wl.SRC_VALUES)
    harness.fill_on_device(dk + dv, w.seed * 16 + wl.DST_VALUES)
    src, dst = Pool(sk, sv), Pool(dk, dv)
    table, _ = wl.request_table(w.seed, shape.num_blocks, w.table_blocks)
    free, _ = wl.free_list(w.seed, shape.num_blocks)
    max_tok = 256
    bits = wl.values16(w.seed, wl.APPEND_VALUES, shape.num_layers * 2 * max_tok * src.slot_bytes // 2, shape.dtype)
    append_pool = torch.from_numpy(bits.view(np.uint8).reshape(shape.num_layers, 2, max_tok, src.slot_bytes)).cuda()
    mig, dec = torch.cuda.Stream(), torch.cuda.Stream()
    out = {"workload": w.name, "layers": shape.num_layers, "kv_heads": shape.kv_heads,
           "head_dim": shape.head_dim, "decode_step_ms": 20.0, "by_len": {}}
    for length in w.lengths:
        log("downtime sweep", length)
        res = []
        for r in range(reps + 1):
            m, dt = migrate.run_timed(src, dst, table, length, free, append_pool, mig, dec, step_ms=20.0)
            if r:
                res.append((m, dt))
        # blocking copy: the whole request as one stage, all of it downtime
        blocking = []
        for r in range(reps + 1):
            mm = migrate.Migration(src, dst, table, free, mig)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            mm.stage(length, final=True, time_it=False)
            mig.synchronize()
            if r:
                blocking.append((time.perf_counter() - t0) * 1e6)
        s1 = [m.stages[0] for m, _ in res]
        s1_us = statistics.median(s.gpu_us for s in s1)
        s1_bytes = stage_bytes(s1[0].blocks, shape, src.tile_bytes)
        out["by_len"][str(length)] = {
            "stages": statistics.median(len(m.stages) for m, _ in res),
            "stage1_blocks": s1[0].blocks,
            "stage1_us": round(s1_us, 1),
            "stage1_GBps": round(s1_bytes / (s1_us * 1e-6) / 1e9, 1),
            "final_blocks": res[0][0].stages[-1].blocks,
            "downtime_us_median": round(statistics.median(dt for _, dt in res), 1),
            "downtime_us_min": round(min(dt for _, dt in res), 1),
            "blocking_copy_downtime_us_median": round(statistics.median(blocking), 1),
        }
    src.close()
    dst.close()
    return out


if __name__ == "__main__":
    main()
