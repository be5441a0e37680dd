#!/usr/bin/env python3
"""Benchmark: cross-mesh resharding throughput on one MI355X.

One step = one reshard_execute of the whole resharding task (one fused
kernel launch reading every unique slice once and writing every destination
shard, replicas included) over inputs already resident in HBM.  Consecutive
steps use distinct sets of source and destination buffers in turn (at least
4 GiB of buffers in all), so no step finds its inputs in the 256 MB
last-level cache from the steps just before it.  The plan (decomposition,
sender choice, lowering) is built once before the timed region, as a
resharding task is planned once and repeated every iteration.  Its cost is
reported separately as plan_us.

Prints ONE JSON line.  Default workload: fp16 [8,2048,12288] (403 MB), source
mesh (4,8) "R R S^{01}" -> destination mesh (4,8) "R S^1 R" (4x replicated),
i.e. 384 MiB read + 1536 MiB written per step.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
METRIC = "effective resharding GB/s (read+write) and % of MI355X HBM peak, 1 GPU"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_counters.json")
SETUP_BLOCK = 128  # workgroup size of the setup and check launches (never the timed plan's default)
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2211_05322_amd", "csrc", f) for f in ("execute.hip", "desc.h", "planner.cpp")]


def kernel_hash():
    """Hash of the kernel and lowering code, comments and blank space removed
    (a comment edit does not invalidate recorded counter traffic)."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def traffic_key(workload_name, flags, strategy):
    return f"{workload_name}|flags={flags}|{strategy}"


def measured_traffic(key, bytes_read, bytes_written):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they
    match this kernel.  A record whose reads or writes fall below the plan's
    algorithmic bytes cannot be the timed launch's (every unique byte is read
    and every replica written once), so it is not reported."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f).get(key)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("kernel_hash") != kernel_hash():
        return None
    if rec.get("fetch_bytes", 0) < bytes_read or rec.get("write_bytes", 0) < bytes_written:
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_baseline(w, src_dev, budget_s):
    """The numpy oracle on host cores, on the same workload (bounded repeat count)."""
    import oracle
    from paper_2211_05322_amd.workloads import as_numpy_bits

    src = [as_numpy_bits(t) for t in src_dev]
    es = src[0].dtype.itemsize
    rd, wr = oracle.traffic_bytes(w.shape, es, w.dst_mesh, w.dst_spec)
    times = []
    t_start = time.perf_counter()
    while True:
        t0 = time.perf_counter()
        out = oracle.reshard(src, w.shape, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec)
        times.append(time.perf_counter() - t0)
        del out
        if time.perf_counter() - t_start >= budget_s or len(times) >= 100:
            break
    med = statistics.median(times)
    ncores = len(os.sched_getaffinity(0))
    return {"value": round((rd + wr) / med / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"full workload, {len(times)} run(s) of unshard+reshard in numpy on raw bits, "
                      f"median {med:.3f} s; 1 thread used of {ncores} host cores; "
                      f"bytes counted as read {rd} + written {wr}"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default=None,
                    help="workload id 1..5 (default 5), uneven5 / uneven3 (workloads 5 / 3 with an uneven last "
                         "dimension), transposed2 / transposed5 (workloads 2 / 5 with the destination stored "
                         "[batch, hidden, seq]), or fanoutR (1 GiB, one sender to R replicas)")
    ap.add_argument("--strategy", choices=["broadcast", "sendrecv", "allgather"], default="broadcast",
                    help="broadcast (default) or a comparison strategy that re-reads slices per receiver")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--chunk-bytes", type=int, default=0)
    ap.add_argument("--max-wgs-per-cu", type=int, default=0,
                    help="resident workgroups per CU (0: the library's choice per kernel; -1: no cap)")
    ap.add_argument("--block-threads", type=int, default=0)
    ap.add_argument("--flags", type=int, default=0)
    ap.add_argument("--buffer-sets", type=int, default=0,
                    help="distinct source/destination buffer sets used in turn (0: enough for 4 GiB; "
                         "1: the same buffers every step)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle timing")
    ap.add_argument("--no-context", action="store_true", help="skip the device copy/fill ceiling")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, run a plain device copy of this many MiB 3 times "
                         "(a known-size kernel for hardware counter calibration)")
    ap.add_argument("--calib-fill-mib", type=int, default=0,
                    help="after timing, fill one buffer of this many MiB 3 times with the HIP runtime's "
                         "hipMemsetD32Async (its write form, for comparison in kernel traces and counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: every mesh device is a buffer on a single MI355X; "
              "resharding across several GPUs is not implemented here (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2211_05322_amd import binding as B
    from paper_2211_05322_amd.workloads import BENCH_WORKLOAD, make_workload_tensor, workload_by_name

    w = workload_by_name(args.config or BENCH_WORKLOAD)
    flags = args.flags | {"broadcast": 0, "sendrecv": B.RESHARD_STRATEGY_SENDRECV,
                          "allgather": B.RESHARD_STRATEGY_ALLGATHER}[args.strategy]
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    B.load()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    # Inputs: the logical tensor is generated on the GPU and laid out on the
    # source mesh by the library itself (a reshard from one buffer).
    x = make_workload_tensor(w, seed=args.seed, device="cuda")
    rep = "".join("R" for _ in w.shape)
    # (setup and check launches use 128-thread workgroups, which every kernel
    # honours, so kernel traces and counter runs tell them apart from the
    # timed launches)
    scatter = B.reshard_plan(w.shape, w.dtype, (1,), rep, w.src_mesh, w.src_spec, block_threads=SETUP_BLOCK,
                             dst_perm=w.src_perm)
    src = B.empty_shards(scatter, 1)
    B.reshard_execute(scatter, [x], src)

    t0 = time.perf_counter()
    plan = B.reshard_plan(w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec,
                          flags=flags, chunk_bytes=args.chunk_bytes, block_threads=args.block_threads,
                          max_wgs_per_cu=args.max_wgs_per_cu, src_perm=w.src_perm, dst_perm=w.dst_perm)
    plan_us = (time.perf_counter() - t0) * 1e6
    st = B.reshard_plan_stats(plan)
    dst = B.empty_shards(plan, 1)
    footprint = sum(t.numel() * t.element_size() for t in src + dst)
    nsets = args.buffer_sets or min(64, args.steps, max(2, -(-(4 << 30) // max(footprint, 1))))
    nsets = max(1, nsets)
    sets = [(src, dst)]
    for _ in range(nsets - 1):
        s2 = B.empty_shards(scatter, 1)
        B.reshard_execute(scatter, [x], s2)
        sets.append((s2, B.empty_shards(plan, 1)))
    torch.cuda.synchronize()
    # pointer arrays built once per set, as a training loop that reshards
    # the same buffers every iteration would keep them
    ptr_sets = [(B.pointer_array(s_), B.pointer_array(d_)) for s_, d_ in sets]

    for k in range(args.warmup):
        B.reshard_execute(plan, *ptr_sets[k % nsets], stream=stream)
    torch.cuda.synchronize()

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    h0 = time.perf_counter()
    ev0.record(stream)
    for k in range(args.steps):
        B.reshard_execute(plan, *ptr_sets[k % nsets], stream=stream)
    ev1.record(stream)
    host_us = (time.perf_counter() - h0) * 1e6 / args.steps
    torch.cuda.synchronize()
    ms_total = ev0.elapsed_time(ev1)
    ms_per_step = ms_total / args.steps

    # Round-trip check through the library: the dst of every set a step
    # wrote -> one buffer must equal x.
    back_plan = B.reshard_plan(w.shape, w.dtype, w.dst_mesh, w.dst_spec, (1,), rep, block_threads=SETUP_BLOCK,
                               src_perm=w.dst_perm)
    back = B.empty_shards(back_plan, 1)
    roundtrip_ok = True
    for _, d_ in sets[:min(nsets, max(args.warmup, args.steps))]:
        B.reshard_execute(back_plan, d_, back)
        torch.cuda.synchronize()
        roundtrip_ok &= bool(torch.equal(back[0].view(torch.uint8), x.view(torch.uint8)))
    del back, sets, ptr_sets, dst

    nbytes = st["bytes_read"] + st["bytes_written"]
    gbs = nbytes / (ms_per_step * 1e-3) / 1e9

    context = None
    if not args.no_context:
        # The same box's plain device copy (read N + write N) and fill (write
        # N) at the reshard's total traffic, timed the same way: context for
        # the roofline fraction, not part of the metric.
        half = (nbytes // 2) & ~4095
        a = torch.empty(half, dtype=torch.uint8, device="cuda")
        c = torch.empty_like(a)

        def _rate(fn, moved):
            fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(10):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            return moved / (e0.elapsed_time(e1) / 10 * 1e-3) / 1e9

        context = {"device_copy_GBps": round(_rate(lambda: c.copy_(a), 2 * half), 1),
                   "device_fill_GBps": round(_rate(lambda: c.fill_(7), half), 1),
                   "bytes_each": half}
        del a, c
    if args.calib_copy_mib:
        n = args.calib_copy_mib << 20
        a = torch.empty(n, dtype=torch.uint8, device="cuda")
        c = torch.empty_like(a)
        torch.cuda.synchronize()
        for _ in range(3):
            c.copy_(a)
        torch.cuda.synchronize()
        del a, c
    if args.calib_fill_mib:
        import ctypes
        hip = ctypes.CDLL("libamdhip64.so")
        hip.hipMemsetD32Async.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p]
        hip.hipMemsetD32Async.restype = ctypes.c_int
        n = args.calib_fill_mib << 20
        c = torch.empty(n, dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        for _ in range(3):
            rc = hip.hipMemsetD32Async(ctypes.c_void_p(c.data_ptr()), 7, n // 4, ctypes.c_void_p(stream.cuda_stream))
            if rc != 0:
                raise RuntimeError(f"hipMemsetD32Async failed ({rc})")
        torch.cuda.synchronize()
        del c
    # the counter record holds the default tuning only
    tuned = args.chunk_bytes or args.block_threads or args.max_wgs_per_cu
    traffic = None if tuned else measured_traffic(traffic_key(w.name, args.flags, args.strategy),
                                                  st["bytes_read"], st["bytes_written"])
    # The dominant kernel: the one that processes most of the plan's chunks
    # (an execute launches the direct, row-gather and realignment kernels for
    # the chunks of each kind the plan holds; most workloads use one).
    n_gather, n_realign = B.reshard_plan_gather_chunks(plan), B.reshard_plan_realign_chunks(plan)
    n_gather_u = B.reshard_plan_unaligned_gather_chunks(plan)
    n_unit = B.reshard_plan_unit_gather_chunks(plan)
    n_transpose = B.reshard_plan_transpose_chunks(plan)
    n_direct = st["n_descriptors"] - n_gather - n_gather_u - n_transpose - n_realign
    n_slot = n_gather_u - n_unit
    kernel = max((n_direct, "reshard_kernel"), (n_gather, "reshard_gather_kernel"),
                 (n_slot, "reshard_gather_u_kernel"), (n_unit, "reshard_gather_unit_kernel"),
                 (n_transpose, "reshard_transpose_kernel"), (n_realign, "reshard_realign_kernel"))[1]
    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {1: "u8", 2: "f16", 4: "f32", 8: "f64"}[x.element_size()] if w.dtype != "bfloat16" else "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name, "shape": list(w.shape), "src_mesh": list(w.src_mesh), "src_spec": w.src_spec,
            "dst_mesh": list(w.dst_mesh), "dst_spec": w.dst_spec, "bytes_read": st["bytes_read"],
            "bytes_written": st["bytes_written"], "unit_tasks": st["n_unit_tasks"],
            "workgroups": st["n_descriptors"], "max_fanout": st["max_fanout"], "strategy": args.strategy,
            "buffer_sets": nsets,
        },
        "pct_of_hbm_peak": round(100.0 * gbs / HBM_PEAK_GBS, 2),
        "roofline": {
            "kernel": kernel, "launches_per_step": sum(1 for n in (n_direct, n_gather, n_slot, n_unit, n_transpose, n_realign) if n)
                                                        + (args.strategy == "allgather" and n_direct > 0),
            "bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
        },
        "context": context,
        "plan_us": round(plan_us, 1),
        "host_us_per_execute": round(host_us, 2),
        "roundtrip_ok": roundtrip_ok,
        "kernel_hash": kernel_hash(),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, src, args.cpu_budget)
    print(json.dumps(out), flush=True)
    if not roundtrip_ok:
        sys.exit(3)


if __name__ == "__main__":
    main()
