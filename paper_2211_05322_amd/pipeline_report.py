"""Pipeline-schedule report: 1F1B vs eager-1F1B (Section 4), host only.

    python -m paper_2211_05322_amd.pipeline_report [--comm-ms C --fwd-ms F]

Prints the iteration latency of eager-1F1B relative to 1F1B for 2, 4 and 8
stages, 2x and 4x as many micro-batches as stages, backward = 2 x forward,
and cross-stage resharding costing c = 0 .. 2 forwards (serial links), as a
markdown table; with --comm-ms/--fwd-ms, also that one setting.
"""

from __future__ import annotations

import argparse

from . import binding as B


def ratio(S, M, f, c):
    l1, p1 = B.reshard_pipeline_simulate(S, M, 0, f, 2 * f, c)
    le, pe = B.reshard_pipeline_simulate(S, M, 1, f, 2 * f, c)
    return l1, le, max(pe[s] - p1[s] for s in range(S))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--comm-ms", type=float, default=None)
    ap.add_argument("--fwd-ms", type=float, default=None)
    a = ap.parse_args()
    cs = [0.0, 0.1, 0.25, 0.5, 1.0, 2.0]
    print("| stages | micro-batches | " + " | ".join(f"c = {c} f" for c in cs) + " | extra live activations |")
    print("|---" * (3 + len(cs)) + "|")
    for S in (2, 4, 8):
        for M in (2 * S, 4 * S):
            cells, extra = [], 0
            for c in cs:
                l1, le, extra = ratio(S, M, 1.0, c)
                cells.append(f"{le / l1:.3f}")
            print(f"| {S} | {M} | " + " | ".join(cells) + f" | {extra} |")
    if a.comm_ms is not None and a.fwd_ms is not None:
        print()
        print(f"forward {a.fwd_ms} ms, backward {2 * a.fwd_ms} ms, resharding {a.comm_ms} ms per transfer:")
        print()
        print("| stages | micro-batches | 1F1B ms | eager-1F1B ms | eager / 1F1B |")
        print("|---|---|---|---|---|")
        for S in (2, 4, 8):
            M = 4 * S
            l1, le, _ = ratio(S, M, a.fwd_ms, a.comm_ms)
            print(f"| {S} | {M} | {l1:.2f} | {le:.2f} | {le / l1:.3f} |")


if __name__ == "__main__":
    main()
