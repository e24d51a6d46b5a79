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
import gc
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
PCIE_GBS = 64.0        # PCIe Gen5 x16, per direction


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def copy_kernel_hash() -> str:
    """sha256 of the copy kernel's sources (its device code and launch
    configuration: csrc/common.h followed by csrc/copy_tiles.h)."""
    import hashlib
    h = hashlib.sha256()
    for name in ("common.h", "copy_tiles.h"):
        h.update(open(os.path.join(ROOT, "paper_2406_03243_amd", "csrc", name), "rb").read())
    return h.hexdigest()


def recorded_traffic(kernel: str):
    """HBM bytes per launch of ``kernel`` from the committed counter summary
    (two rocprofv3 --pmc passes, calibrated against a plain copy), or None
    when the kernel source has changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "copy_tiles_bulk_llama7b_traffic.txt")
    try:
        rec = json.load(open(path))
        now = copy_kernel_hash()
    except (OSError, ValueError):
        return None
    if rec.get("kernel") != kernel or rec.get("kernel_source_sha256") != now:
        return None
    return rec["traffic_bytes_per_launch"]


def bulk_span_rows(tile_bytes: int) -> int:
    """The copy kernel's span (1 KiB rows per wavefront) for a bulk launch:
    the power of two at or above a quarter of the tile, within [2, 32]
    (mirrors the library's launch configuration, for labelling only)."""
    quarter = -(-tile_bytes // 4096)
    span = 2
    while span < 32 and span < quarter:
        span *= 2
    return span


def percentile(xs, q):
    """The q-th percentile (0-100) of xs, linear between order statistics."""
    v = sorted(xs)
    if len(v) == 1:
        return v[0]
    pos = (len(v) - 1) * q / 100.0
    lo = int(pos)
    hi = min(lo + 1, len(v) - 1)
    return v[lo] + (v[hi] - v[lo]) * (pos - lo)


def spread(us):
    """Median, p10 and p90 of a list of durations, rounded."""
    return {"median": round(statistics.median(us), 2), "p10": round(percentile(us, 10), 2),
            "p90": round(percentile(us, 90), 2), "n": len(us)}


def inline_launch(src_blocks: int, dst_blocks: int):
    """(ids mode, pairs per launch) of a pool-to-pool stage with host ids:
    16-bit packed ids, 512 pairs a launch, when both pools have at most
    65536 blocks, else 32-bit ids, 256 a launch (mirrors the library's
    launch configuration, for labelling only)."""
    return (2, 512) if max(src_blocks, dst_blocks) <= 65536 else (1, 256)


def stage_bytes(blocks, shape, tile_bytes):
    """Algorithmic bytes of a stage: every tile read once and written once."""
    return 2 * blocks * shape.num_layers * 2 * tile_bytes


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sections", default="downtime,batched,load,xlayout",
                    help="extra workloads after the main one (comma list of downtime, batched, load, xlayout;"
                         " empty for none)")
    ap.add_argument("--downtime-reps", type=int, default=20)
    ap.add_argument("--no-gc-freeze", action="store_true", help="leave set-up objects to the collector")
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
    from paper_2406_03243_amd import harness, migrate, scenarios

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    # ------------------------------------------------------------------ workload
    su = scenarios.llama7b(dev)
    w, shape, src, dst = su.workload, su.shape, su.src, su.dst
    table, free, counts, appends = su.tables[0], su.free, su.counts, su.appends
    log("allocated", w.name, shape)
    initial = su.lengths[0]
    (mig, dec), overlap = harness.concurrent_streams(2)
    torch.cuda.synchronize()

    def step():
        return migrate.run_scheduled(src, dst, table, free, initial, appends, mig, dec)

    # Long-lived objects (torch, the pools) go to the permanent generation, so
    # that a full collection during the timed steps does not walk them.
    gc.collect()
    if not args.no_gc_freeze:
        gc.freeze()
    collections = {0: 0, 1: 0, 2: 0}

    def on_gc(phase, info):
        if phase == "start":
            collections[info["generation"]] += 1

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    log(f"timing {args.steps} steps")
    runs, marks = [], []
    torch.cuda.synchronize()
    gc.callbacks.append(on_gc)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        runs.append(step())          # each step ends on its final stage's synchronisation
        marks.append(time.perf_counter())
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gc.callbacks.remove(on_gc)
    step_ms = [(b - a) * 1e3 for a, b in zip([t0] + marks[:-1], marks)]

    m0 = runs[0][0]
    blocks_per_step = sum(r.blocks for r in m0.stages)
    bytes_per_step = stage_bytes(blocks_per_step, shape, src.tile_bytes)
    ms_per_step = elapsed / args.steps * 1e3
    value = bytes_per_step / (elapsed / args.steps) / 1e9

    # dominant kernel: the bulk pool-to-pool copy of stage 1, launched on the
    # migration stream; its ids travel in the kernel arguments
    s1_blocks = m0.stages[0].blocks
    ids_mode, per_launch_pairs = inline_launch(src.num_blocks, dst.num_blocks)
    launches = math.ceil(s1_blocks / per_launch_pairs)
    s1_us = [m.stages[0].gpu_us for m, _ in runs]
    s1_avg_us = statistics.fmean(s1_us)
    per_launch_bytes = stage_bytes(s1_blocks, shape, src.tile_bytes) / launches
    per_launch_us = s1_avg_us / launches
    achieved = per_launch_bytes / (per_launch_us * 1e-6) / 1e9
    downtimes = [d for _, d in runs]
    kernel_name = "copy_tiles<0, 0, %d, %d>" % (ids_mode, bulk_span_rows(src.tile_bytes))

    # GPU time of every stage's copy (events around its launches), in extra
    # migrations outside the timed region: within the timed steps only stage
    # 1 carries events, since events around the later stages would add their
    # host work to the step (and to the final stage's downtime).
    extra = []
    for _ in range(max(args.steps, 10)):
        mf, _ = migrate.run_scheduled(src, dst, table, free, initial, appends, mig, dec, time_all=True,
                                      time_final=True)
        extra.append(mf)
    final_gpu = [mf.stages[-1].gpu_us for mf in extra]

    # The same launch on contiguous tiles (block i of every layer tensor to
    # block i, as many blocks as stage 1), outside the timed region: what
    # the scattering of a real block table costs the copy.
    from paper_2406_03243_amd.llmig import llmig_stage
    ident = np.arange(s1_blocks, dtype=np.int32)
    cont_us = []
    for r in range(13):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(mig)
        llmig_stage(src, dst, ident, ident, stream=mig)
        e1.record(mig)
        e1.synchronize()
        if r >= 3:
            cont_us.append(e0.elapsed_time(e1) * 1e3)
    cont_gbs = stage_bytes(s1_blocks, shape, src.tile_bytes) / (statistics.median(cont_us) * 1e-6) / 1e9

    stages = []
    for i, rec in enumerate(m0.stages):
        us = [m.stages[i].gpu_us for m, _ in runs if m.stages[i].gpu_us > 0]
        timed_in = "timed steps"
        if not us:
            us = [mf.stages[i].gpu_us for mf in extra]
            timed_in = "extra migrations after the timed steps"
        b = stage_bytes(rec.blocks, shape, src.tile_bytes)
        entry = {"tokens": [rec.from_tok, rec.to_tok], "blocks": rec.blocks, "bytes": b, "final": rec.final,
                 "gpu_us_median": round(statistics.median(us), 2), "gpu_us": spread(us),
                 "GBps": round(b / (statistics.median(us) * 1e-6) / 1e9, 1),
                 "hbm_frac": round(b / (statistics.median(us) * 1e-6) / 1e9 / HBM_PEAK_GBS, 3), "timed_in": timed_in}
        stages.append(entry)

    result = {
        "metric": "KV migration GB/s (fraction of HBM peak); final-stage downtime us vs seq len",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "step_ms": {"median": round(statistics.median(step_ms), 4), "min": round(min(step_ms), 4),
                    "max": round(max(step_ms), 4), "all": [round(x, 3) for x in step_ms],
                    "gc_collections": {f"gen{g}": n for g, n in collections.items()}},
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
                     "avg_launch_us": round(per_launch_us, 2),
                     "contiguous_tiles_GBps": round(cont_gbs, 1),
                     "scattered_vs_contiguous": round(achieved / cont_gbs, 3)},
        "stages": stages,
        "streams_overlap": overlap,
        # the paper's own figures, from another machine and transport: context only
        "paper_context": {"final_stage_downtime_ms": "about 20-30, near-constant in sequence length",
                          "decode_slowdown_while_migrating": "at most 1%",
                          "setup": "two instances on separate VMs, 4x NVIDIA A10 (PCIe 4.0) each, 64 Gb/s "
                                   "network, KV sent with Gloo through CPU buffers; LLaMA-7B and LLaMA-30B",
                          "source": "Llumnix section 6.2"},
        "final_stage_downtime_us": {"median": round(statistics.median(downtimes), 1),
                                    "min": round(min(downtimes), 1), "max": round(max(downtimes), 1),
                                    "p10": round(percentile(downtimes, 10), 2),
                                    "p90": round(percentile(downtimes, 90), 2), "n": len(downtimes)},
        "final_stage_gpu_us": spread(final_gpu),
    }

    # ------------------------------------------------------------------ CPU oracle baseline
    if not args.no_cpu_baseline:
        from paper_2406_03243_amd.llmig import llmig_plan
        s1 = m0.stages[0]
        ms1, _ = llmig_plan(table, free, s1.length, s1.from_tok, s1.to_tok, src.block_size)
        result["cpu_baseline"] = cpu_baseline(
            src, ms1[:CPU_SAMPLE_PAIRS], shape,
            f"{CPU_SAMPLE_PAIRS} of the {s1.blocks} stage-1 block pairs of {w.name}")

    if args.calibration_copy:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        a.fill_(1)
        for _ in range(2):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    su.close()
    del su, src, dst, appends
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    sections = set(args.sections.split(",")) if args.sections else set()
    if "downtime" in sections:
        result["downtime_vs_len"] = downtime_sweep(args.downtime_reps)
        torch.cuda.empty_cache()
    if "batched" in sections:
        result["batched"] = batched_section(cpu=not args.no_cpu_baseline)
        torch.cuda.empty_cache()
    if "load" in sections:
        result["under_load"] = load_section()
        torch.cuda.empty_cache()
    if "xlayout" in sections:
        result["cross_layout"] = xlayout_section()
        torch.cuda.empty_cache()

    print(json.dumps(result), flush=True)


# CPU baseline: the oracle's block-by-block copy on host snapshots of a sample
# of a stage's block pairs.  The sample holds the mapped source blocks only (a
# compact pool behind an id remap) and a zeroed destination of the same size.
CPU_SAMPLE_PAIRS = 256
CPU_WARMUP_RUNS = 3
CPU_TIMED_RUNS = 5
# Threads of the all-core leg: the process's CPU affinity, capped at the CPU
# share a one-GPU job gets on the GPU machines (16 CPUs), where the affinity
# mask can name the whole host.
CPU_SHARE = 16


def cpu_baseline(src, ids, shape, what):
    """The oracle's per-tile copy of the pairs whose source blocks are
    ``ids``, on host snapshots: one thread, then every CPU of the process's
    share on disjoint slices.  Each leg runs CPU_WARMUP_RUNS untimed runs and
    reports the median of CPU_TIMED_RUNS timed ones; a single-thread run is
    one pass over the sample, an all-core run one pass per thread over each
    thread's slice (the same bytes per thread as one pass over the sample).
    ``value`` is the all-core rate."""
    import numpy as np
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    from oracle import HostPool
    from paper_2406_03243_amd import harness

    ids = np.asarray(ids, np.int32)
    n = len(ids)
    hs = HostPool(harness.snapshot_blocks(src.k, ids), harness.snapshot_blocks(src.v, ids),
                  src.block_size, src.slot_bytes)
    hd = HostPool.zeros(shape.num_layers, n, src.block_size, src.slot_bytes)
    local = np.arange(n, dtype=np.int32)
    orc = oracle.default()
    per_pair = 2 * shape.num_layers * 2 * src.tile_bytes      # read + written

    def leg(threads):
        chunks = np.array_split(local, threads)
        passes = threads if threads > 1 else 1

        def work(c):
            for _ in range(passes):
                orc.copy(hs, hd, c, c)

        rates = []
        with ThreadPoolExecutor(max_workers=threads) as ex:
            for r in range(CPU_WARMUP_RUNS + CPU_TIMED_RUNS):
                t0 = time.perf_counter()
                list(ex.map(work, chunks))
                el = time.perf_counter() - t0
                if r >= CPU_WARMUP_RUNS:
                    rates.append(passes * n * per_pair / el / 1e9)
        return {"value": round(statistics.median(rates), 2), "unit": "GB/s", "cores": threads,
                "runs_GBps": [round(x, 2) for x in rates], "warmup_runs": CPU_WARMUP_RUNS,
                "bytes_per_run": passes * n * per_pair}

    affinity = len(os.sched_getaffinity(0))
    threads = max(1, min(CPU_SHARE, affinity, n))
    single = leg(1)
    multi = leg(threads)
    # the host CPU as the kernel reports it (a virtual machine may report
    # only the brand): name, family/model/stepping and clock of the first CPU
    info = {}
    try:
        for line in open("/proc/cpuinfo"):
            if not line.strip():
                break
            key, _, val = line.partition(":")
            info[key.strip()] = val.strip()
    except OSError:
        pass
    model = info.get("model name", "")
    ident = {k.replace(" ", "_"): info[k] for k in ("cpu family", "model", "stepping", "cpu MHz") if k in info}
    return {"value": multi["value"], "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{what}: all {shape.num_layers} layers, K and V, {n * shape.num_layers * 2} tiles of "
                      f"{src.tile_bytes} B, copied from host snapshots (a compact pool of the mapped blocks) by "
                      f"the oracle's per-tile memcpy; median of {CPU_TIMED_RUNS} runs after {CPU_WARMUP_RUNS} "
                      f"warm-ups per leg",
            "all_cores": multi, "single_thread": single,
            "affinity_cpus": affinity, "nproc": os.cpu_count(), "cpu_share_cap": CPU_SHARE,
            "cpu_model": model, "cpu_id": ident}


def downtime_sweep(reps):
    """Final-stage downtime against sequence length, LLaMA-30B quarter."""
    import torch

    from paper_2406_03243_amd import migrate, scenarios

    su = scenarios.llama30b_quarter()
    shape, src, dst, table, free = su.shape, su.src, su.dst, su.tables[0], su.free
    log("allocated", su.workload.name, shape)
    append_pool = su.extra["append_pool"]
    mig, dec = torch.cuda.Stream(), torch.cuda.Stream()
    out = {"workload": su.workload.name, "layers": shape.num_layers, "kv_heads": shape.kv_heads,
           "head_dim": shape.head_dim, "decode_step_ms": 20.0, "by_len": {}}
    for length in su.lengths:
        log("downtime sweep", length)
        res = []
        for r in range(reps + 1):
            m, dt = migrate.run_timed(src, dst, table, length, free, append_pool, mig, dec, step_ms=20.0)
            if r:
                res.append((m, dt))
        # the final stage's GPU time alone (events around its launch)
        final_gpu = []
        for r in range(reps):
            m, _ = migrate.run_timed(src, dst, table, length, free, append_pool, mig, dec, step_ms=20.0,
                                     time_final=True)
            final_gpu.append(m.stages[-1].gpu_us)
        # blocking copy: the whole request as one stage, all of it downtime
        blocking = []
        for r in range(reps + 1):
            mm = migrate.Migration(src, dst, table, free, mig)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            mm.finish(length)
            if r:
                blocking.append((mm.finished_at - t0) * 1e6)
        s1 = [m.stages[0] for m, _ in res]
        s1_us = statistics.median(s.gpu_us for s in s1)
        s1_bytes = stage_bytes(s1[0].blocks, shape, src.tile_bytes)
        out["by_len"][str(length)] = {
            "stages": statistics.median(len(m.stages) for m, _ in res),
            "stage1_blocks": s1[0].blocks,
            "stage1_us": round(s1_us, 1),
            "stage1_GBps": round(s1_bytes / (s1_us * 1e-6) / 1e9, 1),
            "stage1_hbm_frac": round(s1_bytes / (s1_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 3),
            "final_blocks": res[0][0].stages[-1].blocks,
            "downtime_us_median": round(statistics.median(dt for _, dt in res), 1),
            "downtime_us_min": round(min(dt for _, dt in res), 1),
            "downtime_us": spread([dt for _, dt in res]),
            "final_stage_gpu_us_median": round(statistics.median(final_gpu), 1),
            "final_stage_gpu_us": spread(final_gpu),
            "blocking_copy_downtime_us_median": round(statistics.median(blocking), 1),
            "blocking_copy_downtime_us": spread(blocking),
        }
    su.close()
    return out


def batched_section(reps=20, host_reps=3, chunk_pairs=64, cpu=True):
    """64 requests migrated in one llmig_stage call; the same pairs packed
    into and unpacked from device staging (block fusion's kernels alone);
    and the same pairs through pinned host memory (pack -> host -> unpack,
    chunked, two buffers), then each direction alone."""
    import numpy as np
    import torch

    from paper_2406_03243_amd import harness, migrate, scenarios
    from paper_2406_03243_amd.llmig import llmig_stage

    su = scenarios.batched()
    shape, src, dst = su.shape, su.src, su.dst
    log("allocated", su.workload.name, shape)
    ms, md, _ = migrate.plan_batch(su.tables, su.lengths, su.free, shape.block_size)
    nbytes = stage_bytes(len(ms), shape, src.tile_bytes)
    mig = torch.cuda.Stream()
    for _ in range(3):
        llmig_stage(src, dst, ms, md, stream=mig)
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(mig)
        llmig_stage(src, dst, ms, md, stream=mig)
        e1.record(mig)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e3)
    us = statistics.median(times)
    out = {"workload": su.workload.name, "requests": len(su.tables), "pairs": int(len(ms)),
           "pool_blocks": shape.num_blocks, "bytes": nbytes, "stage_us_median": round(us, 1),
           "stage_us": spread(times),
           "GBps": round(nbytes / (us * 1e-6) / 1e9, 1),
           "hbm_frac": round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 3),
           "lengths": {"min": int(min(su.lengths)), "median": float(statistics.median(su.lengths)),
                       "max": int(max(su.lengths)), "tokens": int(sum(su.lengths))}}
    # block fusion with device staging: the pack and unpack kernels alone,
    # each reading and writing every tile once (HBM-bound)
    from paper_2406_03243_amd.llmig import llmig_pack, llmig_unpack
    one_way_all = len(ms) * shape.num_layers * 2 * src.tile_bytes
    staging = torch.empty(one_way_all, dtype=torch.uint8, device="cuda")
    for name, fn, ids in (("pack", llmig_pack, ms), ("unpack", llmig_unpack, md)):
        pool = src if name == "pack" else dst
        for _ in range(3):
            fn(pool, ids, staging, stream=mig)
        torch.cuda.synchronize()
        t = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(mig)
            fn(pool, ids, staging, stream=mig)
            e1.record(mig)
            torch.cuda.synchronize()
            t.append(e0.elapsed_time(e1) * 1e3)
        gbs = 2 * one_way_all / (statistics.median(t) * 1e-6) / 1e9
        out[f"{name}_device_staging"] = {"bytes": 2 * one_way_all, "us": spread(t), "GBps": round(gbs, 1),
                                         "hbm_frac": round(gbs / HBM_PEAK_GBS, 3)}
        log("batched", name, out[f"{name}_device_staging"])
    del staging
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    chunk_bytes = chunk_pairs * shape.num_layers * 2 * src.tile_bytes
    bufs = [torch.empty(chunk_bytes, dtype=torch.uint8, pin_memory=True) for _ in range(2)]
    dev_bufs = [(torch.empty(chunk_bytes, dtype=torch.uint8, device="cuda"),
                 torch.empty(chunk_bytes, dtype=torch.uint8, device="cuda")) for _ in range(2)]
    (ps, us_), overlap = harness.concurrent_streams(2)
    one_way = len(ms) * shape.num_layers * 2 * src.tile_bytes
    out["host_staged"] = {"chunk_pairs": chunk_pairs, "bytes_each_way": one_way,
                          "bound": "PCIe Gen5 x16, ~64 GB/s per direction", "streams_overlap": overlap}
    for mode, db in (("kernel_pcie", None), ("copy_engine", dev_bufs)):
        host_times = []
        for r in range(host_reps + 1):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            migrate.run_host_staged(src, dst, ms, md, bufs, ps, us_, chunk_pairs, dev_bufs=db)
            torch.cuda.synchronize()
            if r:
                host_times.append(time.perf_counter() - t0)
        ht = statistics.median(host_times)
        out["host_staged"][mode] = {"seconds_median": round(ht, 4), "GBps_each_way": round(one_way / ht / 1e9, 2)}

    # One direction at a time (the link each side of a two-GPU migration
    # would carry alone): every chunk packed into the pinned buffers, then
    # every chunk unpacked from them.
    def one_direction(pack: bool) -> float:
        times = []
        for r in range(host_reps + 1):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for c, lo in enumerate(range(0, len(ms), chunk_pairs)):
                if pack:
                    llmig_pack(src, ms[lo:lo + chunk_pairs], bufs[c % 2], stream=ps)
                else:
                    llmig_unpack(dst, md[lo:lo + chunk_pairs], bufs[c % 2], stream=us_)
            torch.cuda.synchronize()
            if r:
                times.append(time.perf_counter() - t0)
        return statistics.median(times)

    for name, pack in (("pack_to_host_alone", True), ("unpack_from_host_alone", False)):
        t = one_direction(pack)
        gbs = one_way / t / 1e9
        out["host_staged"][name] = {"seconds_median": round(t, 4), "GBps": round(gbs, 2),
                                    "link_frac": round(gbs / PCIE_GBS, 3)}
    log("batched host staged", out["host_staged"])
    if cpu:
        # the oracle on a compact sample of the batched pairs, evenly spaced
        # over the concatenated mapping (so over all 64 requests)
        pick = ms[np.linspace(0, len(ms) - 1, CPU_SAMPLE_PAIRS).astype(np.int64)]
        out["cpu_baseline"] = cpu_baseline(src, pick, shape,
                                           f"{CPU_SAMPLE_PAIRS} of the {len(ms)} batched block pairs "
                                           f"(evenly spaced over the 64 requests)")
    su.close()
    return out


def xlayout_section(reps=20):
    """Stage 1 of the LLaMA-7B migration (512 blocks, 4 GiB each way) between
    pools of different intra-tile layouts: the same tensors registered under
    several layouts, timed per layout pair with events on the stage's stream;
    then the same blocks unpacked from device staging with the conversion."""
    import torch

    from paper_2406_03243_amd import harness, scenarios
    from paper_2406_03243_amd import workloads as wl
    from paper_2406_03243_amd.llmig import (LAYOUT_HCNX, LAYOUT_HDN, LAYOUT_HND, LAYOUT_NHD, Pool, llmig_pack,
                                            llmig_stage, llmig_unpack_layout)

    w = wl.LLAMA7B
    shape = w.shape
    sk, sv = harness.alloc_layers(shape)
    dk, dv = harness.alloc_layers(shape)
    harness.fill_on_device(sk + sv, w.seed * 16 + wl.SRC_VALUES)
    harness.fill_on_device(dk + dv, w.seed * 16 + wl.DST_VALUES)
    table, _ = wl.request_table(w.seed, shape.num_blocks, w.table_blocks, w.src_preoccupied)
    free, _ = wl.free_list(w.seed, shape.num_blocks, w.dst_preoccupied)
    n = w.lengths[0] // shape.block_size
    ms, md = table[:n], free[:n]
    names = {LAYOUT_NHD: "NHD", LAYOUT_HND: "HND", LAYOUT_HCNX: "HCNX", LAYOUT_HDN: "HDN"}
    cases = [((LAYOUT_NHD, LAYOUT_NHD), (LAYOUT_NHD, LAYOUT_NHD)),      # same layout: the tile copy
             ((LAYOUT_NHD, LAYOUT_NHD), (LAYOUT_HND, LAYOUT_HND)),      # chunks move whole
             ((LAYOUT_NHD, LAYOUT_NHD), (LAYOUT_HCNX, LAYOUT_HDN)),     # token-major -> vLLM paged attention
             ((LAYOUT_HCNX, LAYOUT_HDN), (LAYOUT_NHD, LAYOUT_NHD))]     # and back
    nbytes = stage_bytes(n, shape, 2 * shape.block_size * shape.kv_heads * shape.head_dim)
    out = {"workload": w.name, "pairs": int(n), "bytes": nbytes, "cases": []}
    mig = torch.cuda.Stream()
    for sl, dl in cases:
        src, dst = Pool(sk, sv, layouts=sl), Pool(dk, dv, layouts=dl)
        for _ in range(3):
            llmig_stage(src, dst, ms, md, stream=mig)
        torch.cuda.synchronize()
        times = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(mig)
            llmig_stage(src, dst, ms, md, stream=mig)
            e1.record(mig)
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) * 1e3)
        us = statistics.median(times)
        gbs = nbytes / (us * 1e-6) / 1e9
        out["cases"].append({"src": "/".join(names[x] for x in sl), "dst": "/".join(names[x] for x in dl),
                             "stage_us_median": round(us, 1), "stage_us": spread(times), "GBps": round(gbs, 1),
                             "hbm_frac": round(gbs / HBM_PEAK_GBS, 3)})
        log("cross-layout", out["cases"][-1])
        src.close()
        dst.close()
    # the receiving side of block fusion across engines: stage 1 packed from
    # the token-major pool into device staging, then scattered into the
    # vLLM-layout pool with the conversion on the way in (timed alone)
    src = Pool(sk, sv, layouts=(LAYOUT_NHD, LAYOUT_NHD))
    dst = Pool(dk, dv, layouts=(LAYOUT_HCNX, LAYOUT_HDN))
    staging = torch.empty(n * shape.num_layers * 2 * src.tile_bytes, dtype=torch.uint8, device="cuda")
    llmig_pack(src, ms, staging, stream=mig)
    for _ in range(3):
        llmig_unpack_layout(dst, md, staging, src.layouts, stream=mig)
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(mig)
        llmig_unpack_layout(dst, md, staging, src.layouts, stream=mig)
        e1.record(mig)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e3)
    us = statistics.median(times)
    gbs = nbytes / (us * 1e-6) / 1e9
    out["unpack_converting"] = {"staging": "NHD/NHD (device)", "dst": "HCNX/HDN", "stage_us_median": round(us, 1),
                                "stage_us": spread(times), "GBps": round(gbs, 1),
                                "hbm_frac": round(gbs / HBM_PEAK_GBS, 3)}
    log("cross-layout unpack", out["unpack_converting"])
    src.close()
    dst.close()
    del sk, sv, dk, dv, staging
    return out


def load_section(reps=5, reader_passes=3, step_ms=20.0, caps=(0, 256, 64)):
    """GQA long-context migration beside a streaming reader of a separate
    40 GB region (all streams at the default priority), for several caps on
    the migration's copy grid (0: uncapped)."""
    import torch

    from paper_2406_03243_amd import harness, migrate, scenarios
    from paper_2406_03243_amd.llmig import llmig_stream_read

    su = scenarios.gqa_long()
    shape, src, dst, table, free = su.shape, su.src, su.dst, su.tables[0], su.free
    log("allocated", su.workload.name, shape)
    region, append_pool = su.extra["region"], su.extra["append_pool"]
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    wgs = cus * 4
    sink = torch.empty(wgs * 256, dtype=torch.int64, device="cuda")
    (rd, mig, dec), overlap = harness.concurrent_streams(3)
    length = su.lengths[0]
    read_bytes = reader_passes * region.numel() * region.element_size()

    def reader_run():
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(rd)
        llmig_stream_read(region, reader_passes, wgs, sink, stream=rd)
        e1.record(rd)
        return e0, e1

    alone_r = []
    for r in range(reps + 1):
        e = reader_run()
        torch.cuda.synchronize()
        if r:
            alone_r.append(e[0].elapsed_time(e[1]) * 1e3)
    r_alone = statistics.median(alone_r)
    out = {"workload": su.workload.name, "tokens": length, "reader_bytes": read_bytes, "streams_overlap": overlap,
           "reader_workgroups": wgs, "reader_alone_GBps": round(read_bytes / (r_alone * 1e-6) / 1e9, 1),
           "by_cap": {}}
    out["beside_decode"] = decode_overhead(su, caps, step_ms)
    for cap in caps:
        alone_m = []
        for r in range(reps + 1):
            m, dt = migrate.run_timed(src, dst, table, length, free, append_pool, mig, dec, step_ms=step_ms,
                                      max_workgroups=cap)
            if r:
                alone_m.append((m, dt))
        both = []
        for r in range(reps + 1):
            torch.cuda.synchronize()
            e = reader_run()
            t0 = time.perf_counter()
            m, dt = migrate.run_timed(src, dst, table, length, free, append_pool, mig, dec, step_ms=step_ms,
                                      max_workgroups=cap)
            t_mig = time.perf_counter() - t0
            torch.cuda.synchronize()
            if r:
                both.append((e[0].elapsed_time(e[1]) * 1e3, m, dt, t_mig))
        r_both = statistics.median(b[0] for b in both)
        t_mig = statistics.median(b[3] for b in both) * 1e6
        s1_bytes = stage_bytes(alone_m[0][0].stages[0].blocks, shape, src.tile_bytes)
        s1_alone = statistics.median(m.stages[0].gpu_us for m, _ in alone_m)
        s1_both = statistics.median(b[1].stages[0].gpu_us for b in both)
        out["by_cap"][str(cap) if cap else "uncapped"] = {
            "reader_with_migration_GBps": round(read_bytes / (r_both * 1e-6) / 1e9, 1),
            "reader_slowdown_during_migration": round(max(0.0, r_both - r_alone) / t_mig, 3),
            "migration_wall_us": round(t_mig, 1),
            "stage1_GBps_alone": round(s1_bytes / (s1_alone * 1e-6) / 1e9, 1),
            "stage1_hbm_frac_alone": round(s1_bytes / (s1_alone * 1e-6) / 1e9 / HBM_PEAK_GBS, 3),
            "stage1_GBps_under_load": round(s1_bytes / (s1_both * 1e-6) / 1e9, 1),
            "stages_under_load": statistics.median(len(b[1].stages) for b in both),
            "downtime_us_alone": round(statistics.median(dt for _, dt in alone_m), 1),
            "downtime_us_under_load": round(statistics.median(b[2] for b in both), 1)}
    su.close()
    return out


def decode_overhead(su, caps, step_ms, steps=14, reps=5):
    """Per-step decode attention time on the source instance (a batch of
    16 requests plus the migrating one, all 80 layers) with and without a
    migration running beside it (Llumnix §6.2 reports at most 1% slowdown)."""
    import torch

    from paper_2406_03243_amd import harness, migrate, scenarios
    from paper_2406_03243_amd.llmig import decode_workspace_bytes, llmig_decode_attention

    shape, src, dst, table, free = su.shape, su.src, su.dst, su.tables[0], su.free
    append_pool = su.extra["append_pool"]
    tables, ctx, q = scenarios.decode_batch(su)
    out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    ws = torch.empty(decode_workspace_bytes(ctx, shape.num_layers, q.shape[2], shape.head_dim),
                     dtype=torch.uint8, device="cuda")
    scale = 1.0 / math.sqrt(shape.head_dim)
    (at, mig, dec), overlap = harness.concurrent_streams(3)
    kv_bytes = sum(ctx) * shape.num_layers * 2 * shape.kv_heads * shape.head_dim * shape.elem_bytes

    def decode_steps(n):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
        evs[0].record(at)
        for i in range(n):
            llmig_decode_attention(src, q, tables, ctx, scale, ws, out, stream=at)
            evs[i + 1].record(at)
        return evs

    for _ in range(3):
        llmig_decode_attention(src, q, tables, ctx, scale, ws, out, stream=at)
    torch.cuda.synchronize()
    evs = decode_steps(steps)
    torch.cuda.synchronize()
    alone = [evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(steps)]
    t_alone = statistics.median(alone)
    res = {"batch": len(ctx), "tokens": int(sum(ctx)), "kv_bytes_per_step": kv_bytes, "streams_overlap": overlap,
           "step_us_alone": round(t_alone, 1), "decode_GBps_alone": round(kv_bytes / (t_alone * 1e-6) / 1e9, 1),
           "by_cap": {}}
    for cap in caps:
        rows = []
        for r in range(reps):
            torch.cuda.synchronize()
            evs = decode_steps(steps)
            m0 = torch.cuda.Event(enable_timing=True)
            m1 = torch.cuda.Event(enable_timing=True)
            # let two decode steps run, then start the migration beside them
            mig.wait_event(evs[2])
            m0.record(mig)
            m, dt = migrate.run_timed(src, dst, table, su.lengths[0], free, append_pool, mig, dec,
                                      step_ms=step_ms, max_workgroups=cap)
            m1.record(mig)
            torch.cuda.synchronize()
            start, stop = evs[0].elapsed_time(m0), evs[0].elapsed_time(m1)
            over = [evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(steps)
                    if evs[0].elapsed_time(evs[i + 1]) > start and evs[0].elapsed_time(evs[i]) < stop]
            rows.append((over, (stop - start) * 1e3, dt))
        over = [x for o, _, _ in rows for x in o]
        res["by_cap"][str(cap) if cap else "uncapped"] = {
            "migration_us": round(statistics.median(r[1] for r in rows), 1),
            "overlapping_steps": round(statistics.mean(len(r[0]) for r in rows), 1),
            "extra_decode_us_per_migration": round(statistics.median(sum(x - t_alone for x in r[0])
                                                                     for r in rows), 1),
            "step_us_during_migration_mean": round(statistics.mean(over), 1),
            "step_us_during_migration_max": round(max(over), 1),
            "decode_slowdown_during_migration": round(statistics.mean(over) / t_alone - 1, 3),
            "downtime_us": round(statistics.median(r[2] for r in rows), 1)}
    res["carried"] = carried_overhead(su, q, tables, ctx, scale, ws, out, at, mig, dec, steps, reps, t_alone)
    return res


def carried_overhead(su, q, tables, ctx, scale, ws, out, at, mig, dec, steps, reps, t_alone, splits=(1, 4)):
    """The same migration with its first stage carried by decode steps
    (llmig_decode_attention_migrate): `split` consecutive steps of the
    batch, the migrating request among their sequences, write its whole
    blocks into the destination as their attention reads them; each step
    adds the request's next token, and once the host has seen the last
    carrying step complete, the final stage copies the rest beside the
    steps that follow.  The decode time this costs is the carrying steps'
    excess over a step alone, plus that of any step the final stage ran
    beside."""
    import torch

    from paper_2406_03243_amd import migrate
    from paper_2406_03243_amd.llmig import (llmig_decode_attention, llmig_decode_attention_migrate,
                                            llmig_write_tokens)

    src, dst, table, free = su.src, su.dst, su.tables[0], su.free
    seq, initial = len(ctx) - 1, su.lengths[0]
    append_pool = su.extra["append_pool"]
    out_rows = {}
    for split in splits:
        rows = []
        for r in range(reps):
            m = migrate.Migration(src, dst, table, free, mig)
            rec, _, md = m.plan(initial, final=False)
            with torch.cuda.stream(at):
                ids = torch.from_numpy(md).to("cuda")
            bounds = [len(md) * k // split for k in range(split + 1)]
            torch.cuda.synchronize()
            evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
            evs[0].record(at)
            for i in range(steps):
                k = i - 2
                if 0 <= k < split:
                    llmig_decode_attention_migrate(src, q, tables, ctx, scale, ws, out, dst, seq,
                                                   ids[bounds[k]:bounds[k + 1]], bounds[k], stream=at)
                else:
                    llmig_decode_attention(src, q, tables, ctx, scale, ws, out, stream=at)
                evs[i + 1].record(at)
            # each carrying step's token, written by decode
            with torch.cuda.stream(dec):
                data = append_pool[:, :, :split].contiguous()
            dec.wait_event(evs[2])
            llmig_write_tokens(src, table, initial, data, stream=dec)
            evs[2 + split].synchronize()
            dec.synchronize()
            t0 = time.perf_counter()
            m.finish(initial + split)
            downtime = (m.finished_at - t0) * 1e6
            m1 = torch.cuda.Event(enable_timing=True)
            m1.record(mig)
            torch.cuda.synchronize()
            stop = evs[0].elapsed_time(m1)
            st = [evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(steps)]
            over = [st[i] for i in range(2, steps) if i < 2 + split or evs[0].elapsed_time(evs[i]) < stop]
            rows.append((st[2:2 + split], over, downtime))
            m.abort()
        carried = [x for c, _, _ in rows for x in c]
        out_rows[f"split_{split}"] = {
            "carrying_steps": split,
            "stage_bytes_written": int(len(md) * su.shape.num_layers * 2 * src.tile_bytes),
            "carrying_step_us_mean": round(statistics.mean(carried), 1),
            "carrying_step_slowdown": round(statistics.mean(carried) / t_alone - 1, 3),
            "extra_decode_us_per_migration": round(statistics.median(sum(x - t_alone for x in o)
                                                                     for _, o, _ in rows), 1),
            "overlapping_steps": round(statistics.mean(len(o) for _, o, _ in rows), 1),
            "downtime_us": round(statistics.median(d for _, _, d in rows), 1)}
    out_rows["split_1_final_carried"] = carried_final_overhead(su, q, tables, ctx, scale, out, at, dec, steps, reps,
                                                               t_alone)
    return out_rows


def carried_final_overhead(su, q, tables, ctx, scale, out, at, dec, steps, reps, t_alone):
    """Both stages carried: step 2 of the batch carries stage 0 (every
    whole block of the migrating request) and produces the request's next
    token, which decode writes into its partly filled last block; step 3,
    the request's last on the source, reads that token too and carries the
    final stage (that block).  Once step 3 is over the destination holds the
    whole request, so nothing is copied after it leaves the batch: no
    downtime beyond the step.  The decode time this costs is the two
    carrying steps' excess over a step alone."""
    import torch

    from paper_2406_03243_amd import migrate
    from paper_2406_03243_amd.llmig import (decode_workspace_bytes, llmig_decode_attention,
                                            llmig_decode_attention_migrate, llmig_write_tokens)

    src, dst, table, free = su.src, su.dst, su.tables[0], su.free
    seq, initial, bs = len(ctx) - 1, su.lengths[0], su.shape.block_size
    ctx1 = list(ctx)
    ctx1[seq] = initial + 1                       # the request after step 2's token
    ws1 = torch.empty(decode_workspace_bytes(ctx1, su.shape.num_layers, q.shape[2], su.shape.head_dim),
                      dtype=torch.uint8, device="cuda")
    with torch.cuda.stream(dec):
        data = su.extra["append_pool"][:, :, :1].contiguous()
    rows = []
    for r in range(reps):
        m = migrate.Migration(src, dst, table, free, at)       # plans only: the steps carry the copies
        rec0, _, md0 = m.plan(initial, final=False)
        rec1, _, md1 = m.plan(initial + 1, final=True)
        with torch.cuda.stream(at):
            ids0 = torch.from_numpy(md0).to("cuda")
            ids1 = torch.from_numpy(md1).to("cuda")
        torch.cuda.synchronize()
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        written = torch.cuda.Event()
        evs[0].record(at)
        for i in range(steps):
            if i == 2:
                llmig_decode_attention_migrate(src, q, tables, ctx, scale, ws1, out, dst, seq, ids0,
                                               rec0.from_tok // bs, stream=at)
            elif i == 3:
                at.wait_event(written)            # the token step 2 produced
                llmig_decode_attention_migrate(src, q, tables, ctx1, scale, ws1, out, dst, seq, ids1,
                                               rec1.from_tok // bs, stream=at)
            else:
                llmig_decode_attention(src, q, tables, ctx if i < 3 else ctx1, scale, ws1, out, stream=at)
            evs[i + 1].record(at)
            if i == 2:
                dec.wait_event(evs[3])
                llmig_write_tokens(src, table, initial, data, stream=dec)
                written.record(dec)
        torch.cuda.synchronize()
        st = [evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(steps)]
        plain_after = statistics.median(st[5:])
        rows.append((st[2], st[3], plain_after))
        m.abort()
    return {"carrying_steps": 2, "final_stage_blocks": len(md1),
            "stage0_step_us_mean": round(statistics.mean(r[0] for r in rows), 1),
            "final_step_us_mean": round(statistics.mean(r[1] for r in rows), 1),
            "plain_step_us_after": round(statistics.mean(r[2] for r in rows), 1),
            "extra_decode_us_per_migration": round(statistics.median(r[0] + r[1] - 2 * t_alone for r in rows), 1),
            "downtime_us": 0.0,
            "downtime_note": "the final stage completes with the request's last decode step on the source"}


if __name__ == "__main__":
    main()
