"""Per-workload report: every resharding workload timed on one GPU.

    python -m paper_2211_05322_amd.workload_report [--steps 50] [--flush-steps 20] [--flush-mib 1024]

For each workload (the five resharding tasks, workloads 5 and 3 with an
uneven last dimension, misaligned rows that arrive in runs, workloads 2 and 5
with the destination buffers transposed, then the one-sender replication
microbenchmark at 1, 4 and 8 receivers) prints one
markdown row: unit tasks, fan-out, chunks per kernel, bytes moved (read +
write), planning time, and four timings of `reshard_execute`:

* back-to-back: mean of `--steps` consecutive launches on one set of
  buffers (HIP events on the launch stream around all of them), the way
  `bench.py` times;
* rotated: the same over several distinct sets of source and destination
  buffers, used in turn, with at least 4 GiB of buffers in all, so a launch
  finds nothing of its own inputs in the 256 MB last-level cache (MALL) from
  the launches just before it;
* cold: mean of `--flush-steps` launches, each preceded by a read-only pass
  over a `--flush-mib` scratch buffer (clean lines only, so the launch pays
  no write-back of someone else's data), HIP events around each launch;
* graph: the back-to-back buffers, 50 executes captured into one HIP graph
  (after `reshard_plan_upload`) and replayed, per reshard: what a caller
  that replays its resharding saves on launch overhead.

Each row ends with a round-trip check through the library (destination back
to one buffer, compared bit for bit with the generated tensor).

Each workload runs in a process of its own (as `bench.py` does), started by a
parent that never touches the GPU: after other workloads' buffers have come
and gone in the same process, the same launch measured up to 2 % slower on
one machine (workload 5 rotated: 361.0 us alone, 366.2 us after workloads
1-4).  `--one-process` keeps them in one process.
"""

from __future__ import annotations

import argparse
import subprocess
import sys
import time

import torch

from . import binding as B
from .workloads import make_workload_tensor, workload_by_name

HBM_PEAK_GBS = 8000.0


def _time_back_to_back(fn, steps, stream):
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / steps


def _time_graph(plan, sp, dp, per_graph=50, replays=10):
    B.reshard_plan_upload(plan)  # the upload stays outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(per_graph):
            B.reshard_execute(plan, sp, dp)
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(replays):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    del g
    return e0.elapsed_time(e1) * 1e3 / (per_graph * replays)


def _time_cold(fn, steps, scratch, stream):
    evs = []
    for k in range(steps):
        scratch.sum()  # reads the whole buffer, writes one word
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        evs.append((e0, e1))
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in evs) * 1e3 / steps


def report_row(key, w, steps, flush_steps, scratch, stream):
    x = make_workload_tensor(w, seed=0, device="cuda")
    rep = "R" * len(w.shape)
    # setup and check plans run 128-thread workgroups (told apart from the
    # timed plan's in kernel traces)
    scatter = B.reshard_plan(w.shape, w.dtype, (1,), rep, w.src_mesh, w.src_spec, block_threads=128,
                             dst_perm=w.src_perm)
    src = B.empty_shards(scatter, 1)
    B.reshard_execute(scatter, [x], src)
    t0 = time.perf_counter()
    plan = B.reshard_plan(w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec, src_perm=w.src_perm,
                          dst_perm=w.dst_perm)
    plan_ms = (time.perf_counter() - t0) * 1e3
    st = B.reshard_plan_stats(plan)
    n_gather, n_realign = B.reshard_plan_gather_chunks(plan), B.reshard_plan_realign_chunks(plan)
    n_gather_u = B.reshard_plan_unaligned_gather_chunks(plan)
    n_transpose = B.reshard_plan_transpose_chunks(plan)
    n_direct = st["n_descriptors"] - n_gather - n_gather_u - n_transpose - n_realign
    dst = B.empty_shards(plan, 1)
    sp0, dp0 = B.pointer_array(src), B.pointer_array(dst)  # built once, as a caller's loop would
    run = lambda: B.reshard_execute(plan, sp0, dp0, stream=stream)  # noqa: E731
    for _ in range(5):
        run()
    torch.cuda.synchronize()
    warm_us = _time_back_to_back(run, steps, stream)
    cold_us = _time_cold(run, flush_steps, scratch, stream)
    graph_us = _time_graph(plan, sp0, dp0)
    # rotated: distinct buffer sets in turn
    footprint = sum(t.numel() * t.element_size() for t in src + dst)
    nsets = min(64, max(2, -(-(4 << 30) // max(footprint, 1))))
    sets = [(src, dst)]
    for _ in range(nsets - 1):
        s2 = B.empty_shards(scatter, 1)
        B.reshard_execute(scatter, [x], s2)
        sets.append((s2, B.empty_shards(plan, 1)))
    ptrs = [(B.pointer_array(s_), B.pointer_array(d_)) for s_, d_ in sets]
    cur = [0]

    def run_rot():
        sp, dp = ptrs[cur[0] % nsets]
        cur[0] += 1
        B.reshard_execute(plan, sp, dp, stream=stream)

    for _ in range(nsets):
        run_rot()
    torch.cuda.synchronize()
    rot_us = _time_back_to_back(run_rot, max(steps, 2 * nsets), stream)
    del sets, ptrs
    back_plan = B.reshard_plan(w.shape, w.dtype, w.dst_mesh, w.dst_spec, (1,), rep, block_threads=128,
                               src_perm=w.dst_perm)
    back = B.empty_shards(back_plan, 1)
    B.reshard_execute(back_plan, dst, back)
    torch.cuda.synchronize()
    ok = bool(torch.equal(back[0].view(torch.uint8), x.view(torch.uint8)))
    moved = st["bytes_read"] + st["bytes_written"]
    gbs = lambda us: moved / us / 1e3  # noqa: E731
    n_unit = B.reshard_plan_unit_gather_chunks(plan)
    kinds = "/".join(str(n) for n in (n_direct, n_gather, n_gather_u - n_unit, n_unit, n_transpose, n_realign))
    row = (f"| {key} | {w.name} | {st['n_unit_tasks']} | {st['max_fanout']} | {kinds} | {moved / 1e6:.1f} | "
           f"{plan_ms:.2f} | {warm_us:.1f} | {100 * gbs(warm_us) / HBM_PEAK_GBS:.1f} | "
           f"{rot_us:.1f} ({nsets}) | {100 * gbs(rot_us) / HBM_PEAK_GBS:.1f} | "
           f"{cold_us:.1f} | {100 * gbs(cold_us) / HBM_PEAK_GBS:.1f} | "
           f"{'bit-exact' if ok else 'MISMATCH'} | {graph_us:.1f} |")
    del x, src, dst, back
    torch.cuda.empty_cache()
    return row, ok


def _print_header():
    print("| id | workload | unit tasks | fan-out | chunks direct/gather/unaligned gather (slots/units)/transpose/realign | MB moved | "
          "plan ms | "
          "back-to-back µs | % | rotated µs (n) | % | cold µs | % | round trip | graph µs |")
    print("|---" * 15 + "|", flush=True)  # (the chunks column lists six counts)


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--flush-steps", type=int, default=20)
    ap.add_argument("--flush-mib", type=int, default=1024)
    ap.add_argument("--workloads", default="1,2,3,4,5,uneven5,uneven3,uneven5_1rep,runs1,runs2,runs4,transposed2,transposed5,"
                                           "fanout1,fanout4,fanout8")
    ap.add_argument("--one-process", action="store_true", help="run every workload in this process")
    ap.add_argument("--rows-only", action="store_true", help=argparse.SUPPRESS)  # a child of the isolating parent
    a = ap.parse_args()
    keys = a.workloads.split(",")
    if not a.one_process and not a.rows_only:
        # one child per workload; this process never initialises the GPU
        print(f"One process per workload; back-to-back: mean of {a.steps} launches; rotated: the same over (n) "
              f"buffer sets in turn; cold: mean of {a.flush_steps} launches, each after a read of {a.flush_mib} "
              f"MiB; graph: per reshard, 50 captured executes replayed; % of {HBM_PEAK_GBS:.0f} GB/s\n")
        _print_header()
        failed = False
        for key in keys:
            r = subprocess.run([sys.executable, "-m", "paper_2211_05322_amd.workload_report", "--rows-only",
                                "--steps", str(a.steps), "--flush-steps", str(a.flush_steps),
                                "--flush-mib", str(a.flush_mib), "--workloads", key])
            if r.returncode != 0:
                failed = True
                if r.returncode != 3:  # 3: a round-trip mismatch, reported in the row
                    raise SystemExit(f"workload {key}: exit status {r.returncode}")
        if failed:
            raise SystemExit(3)
        return
    if not torch.cuda.is_available():
        raise SystemExit("no GPU visible")
    B.load()
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    scratch = torch.ones((a.flush_mib << 20) // 4, dtype=torch.int32, device="cuda")
    if not a.rows_only:
        print(f"{torch.cuda.get_device_name(0)}; back-to-back: mean of {a.steps} launches; rotated: the same "
              f"over (n) buffer sets in turn; cold: mean of {a.flush_steps} launches, each after a read of "
              f"{a.flush_mib} MiB; graph: per reshard, 50 captured executes replayed; % of "
              f"{HBM_PEAK_GBS:.0f} GB/s\n")
        _print_header()
    all_ok = True
    for key in keys:
        w = workload_by_name(key)
        row, ok = report_row(key, w, a.steps, a.flush_steps, scratch, stream)
        all_ok &= ok
        print(row, flush=True)
    if not all_ok:
        raise SystemExit(3)


if __name__ == "__main__":
    main()
