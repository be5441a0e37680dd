"""Overlap of resharding with computation on one GPU (the premise of Section 4).

    python -m paper_2211_05322_amd.overlap_report [--n 8192] [--reps 20]

The pipeline schedules of Section 4 overlap cross-stage resharding with
the stages' computation.  On one MI355X both share the chip, so this
measures how much of a reshard hides under a compute-bound kernel: an
n x n x n bf16 matrix product (torch.matmul on contiguous operands) on one
stream and the benchmark's reshard (fp16 [8,2048,12288], (4,8) -> (4,8),
4x replicated) on another.  Prints, as a markdown table, each alone,
both in sequence on one stream and both concurrently on two streams (HIP
events around `--reps` repetitions), and the overlap: the fraction of the
shorter operation that disappears when they run together.
"""

from __future__ import annotations

import argparse

import torch

from . import binding as B
from .workloads import BENCH_WORKLOAD, WORKLOADS, make_workload_tensor


def _timed(fn, reps):
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps  # ms, on the current stream's timeline


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--n", type=int, default=8192)
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--max-wgs-per-cu", type=int, default=0,
                    help="the reshard's residency cap (0: the library's; -1: none, so it reserves no LDS)")
    a = ap.parse_args()
    if not torch.cuda.is_available():
        raise SystemExit("no GPU visible")
    B.load()
    torch.cuda.set_device(0)
    w = WORKLOADS[BENCH_WORKLOAD]
    x = make_workload_tensor(w, seed=0, device="cuda")
    rep = "R" * len(w.shape)
    scatter = B.reshard_plan(w.shape, w.dtype, (1,), rep, w.src_mesh, w.src_spec, block_threads=1024)
    src = B.empty_shards(scatter, 1)
    B.reshard_execute(scatter, [x], src)
    plan = B.reshard_plan(w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec,
                          max_wgs_per_cu=a.max_wgs_per_cu)
    dst = B.empty_shards(plan, 1)
    g = torch.Generator(device="cuda").manual_seed(0)
    A = torch.randn((a.n, a.n), generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    Bm = torch.randn((a.n, a.n), generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    C = torch.empty((a.n, a.n), device="cuda", dtype=torch.bfloat16)
    s_comm = torch.cuda.Stream()
    main_stream = torch.cuda.current_stream()

    def gemm():
        torch.matmul(A, Bm, out=C)

    def reshard(stream=None):
        B.reshard_execute(plan, src, dst, stream=stream)

    for _ in range(3):
        gemm()
        reshard()
    t_gemm = _timed(gemm, a.reps)
    t_resh = _timed(reshard, a.reps)
    t_seq = _timed(lambda: (gemm(), reshard()), a.reps)

    def both():
        s_comm.wait_stream(main_stream)
        reshard(s_comm)
        gemm()
        main_stream.wait_stream(s_comm)

    t_par = _timed(both, a.reps)
    hidden = (t_gemm + t_resh - t_par) / min(t_gemm, t_resh)
    flops = 2.0 * a.n ** 3
    st = B.reshard_plan_stats(plan)
    moved = st["bytes_read"] + st["bytes_written"]
    cap = {0: "the library's residency cap", -1: "no residency cap"}.get(a.max_wgs_per_cu,
                                                                     f"{a.max_wgs_per_cu} workgroups per CU")
    print(f"{torch.cuda.get_device_name(0)}; {a.reps} repetitions; reshard with {cap}; ms per repetition\n")
    print("| work | ms | rate |")
    print("|---|---|---|")
    print(f"| bf16 matmul {a.n}³ alone | {t_gemm:.3f} | {flops / t_gemm / 1e9:.0f} TFLOP/s |")
    print(f"| reshard {w.name} alone | {t_resh:.3f} | {moved / t_resh / 1e6:.0f} GB/s |")
    print(f"| both, one stream (sequential) | {t_seq:.3f} | |")
    print(f"| both, two streams (overlapped) | {t_par:.3f} | |")
    print(f"\noverlap: {100 * hidden:.0f} % of the shorter operation is hidden "
          f"((alone + alone − together) / shorter)")


if __name__ == "__main__":
    main()
