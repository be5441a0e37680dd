"""Scheduling report: the Section 3.2 algorithms on the Table 3 cases.

    python -m paper_2211_05322_amd.schedule_report [--dtype float16] [--budget N] [--rounds N]

For every case (a node = a mesh row) prints the number of unit tasks, the
makespan of each algorithm divided by the per-host lower bound, and the host
time each algorithm takes (median of 5 calls), as a markdown table.  Host only.
"""

from __future__ import annotations

import argparse
import statistics
import time

from . import binding as B
from .workloads import TABLE3_CASES, TABLE3_SHAPE

ALGOS = ["naive", "load_balance", "dfs", "randomized", "ensemble"]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--dtype", default="float16")
    ap.add_argument("--budget", type=int, default=200000, help="DFS branch budget")
    ap.add_argument("--rounds", type=int, default=16, help="random orders per step")
    ap.add_argument("--seed", type=int, default=0)
    a = ap.parse_args()
    print(f"tensor {TABLE3_SHAPE} {a.dtype}; DFS budget {a.budget} branches; {a.rounds} random orders per step\n")
    print("| case | send → recv | tasks | plan µs | " + " | ".join(f"{x} (span/LB, µs)" for x in ALGOS) + " |")
    print("|---" * (4 + len(ALGOS)) + "|")
    for case, ss, ds, sm, dm in TABLE3_CASES:
        t0 = time.perf_counter()
        p = B.reshard_plan(TABLE3_SHAPE, a.dtype, sm, ss, dm, ds)
        plan_us = (time.perf_counter() - t0) * 1e6
        n = B.reshard_plan_stats(p)["n_unit_tasks"]
        cells = []
        for algo in ALGOS:
            times, r = [], None
            for _ in range(5):
                t0 = time.perf_counter()
                r = B.reshard_schedule(p, sm[-1], dm[-1], algo, max_dfs_nodes=a.budget,
                                       random_rounds=a.rounds, seed=a.seed)
                times.append((time.perf_counter() - t0) * 1e6)
            cells.append(f"{r['makespan'] / r['lower_bound']:.2f}, {statistics.median(times):.0f}")
        print(f"| {case} | {ss} {sm} → {ds} {dm} | {n} | {plan_us:.0f} | " + " | ".join(cells) + " |")


if __name__ == "__main__":
    main()
