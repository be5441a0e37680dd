"""Oracle for the pipeline schedules of Section 4 -- test infrastructure.

Timing model: S stages and M micro-batches; each stage runs its operations
in its schedule's order.  The warm-up of Section 4: with stages numbered
from 1, stage i runs #stages - i + 1 forwards before its first backward under
1F1B and 2(#stages - i) + 1 under eager-1F1B (never more than M); then it
alternates one backward and one forward, then finishes the backwards.  A
forward of micro-batch m on stage i needs stage i-1's forward of m and the
transfer of its activation; a backward needs stage i+1's backward of m and
the transfer of its gradient; the last stage's backward follows its own
forward.  Transfers take a fixed time, overlap with computation and, on a
serial link, go one at a time per directed stage pair in micro-batch order.

Times are computed by the definition, recursively: an operation starts at
the later of its stage's previous finish and its input's arrival.
"""

import functools
import sys


def stage_ops(S, M, s, eager):
    """Operation list of stage s (0-based): ("F"|"B", micro-batch)."""
    i = s + 1
    w = 2 * (S - i) + 1 if eager else S - i + 1
    w = min(w, M)
    ops = [("F", m) for m in range(w)]
    nf, nb = w, 0
    while nf < M:
        ops.append(("B", nb))
        nb += 1
        ops.append(("F", nf))
        nf += 1
    ops += [("B", m) for m in range(nb, M)]
    return ops


def simulate(S, M, eager, f, b, cf, cb, serial=True):
    """Returns (latency, peak live micro-batches per stage)."""
    ops = [stage_ops(S, M, s, eager) for s in range(S)]
    index = [{op: k for k, op in enumerate(ops[s])} for s in range(S)]
    old = sys.getrecursionlimit()
    sys.setrecursionlimit(max(old, 20 * S * M + 1000))
    try:
        @functools.lru_cache(maxsize=None)
        def finish(s, k):
            kind, m = ops[s][k]
            prev = finish(s, k - 1) if k > 0 else 0.0
            return max(prev, ready(s, kind, m)) + (f if kind == "F" else b)

        def done(s, kind, m):
            return finish(s, index[s][(kind, m)])

        @functools.lru_cache(maxsize=None)
        def arrive_f(s, m):  # activation of m reaches stage s from s-1
            start = done(s - 1, "F", m)
            if serial and m > 0:
                start = max(start, arrive_f(s, m - 1))
            return start + cf

        @functools.lru_cache(maxsize=None)
        def arrive_b(s, m):  # gradient of m reaches stage s from s+1
            start = done(s + 1, "B", m)
            if serial and m > 0:
                start = max(start, arrive_b(s, m - 1))
            return start + cb

        def ready(s, kind, m):
            if kind == "F":
                return 0.0 if s == 0 else arrive_f(s, m)
            return done(s, "F", m) if s == S - 1 else arrive_b(s, m)

        latency = max(finish(s, len(ops[s]) - 1) for s in range(S))
    finally:
        sys.setrecursionlimit(old)
    peaks = []
    for s in range(S):
        live = peak = 0
        for kind, _ in ops[s]:
            live += 1 if kind == "F" else -1
            peak = max(peak, live)
        peaks.append(peak)
    return latency, peaks
