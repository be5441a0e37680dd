"""Unit-task scheduling (Section 3.2): oracle pins, then the library's
scheduler checked against facts that do not depend on how either is written.

Oracle pins: exhaustive search over sender assignments and orders on small
task sets (DFS without a budget must reach it; every algorithm must be valid
and no better than it; the lower bound no worse); hand-computed start times
of the per-host-order reduction; Eq. 4's greedy against the exhaustive Eq. 4
minimum where the greedy is exact; the statements of Section 5.3.1 on the
Table 3 cases.

Library (reshard_schedule, C++): every schedule is valid under Eq. 2-3 and
its makespan is Eq. 1 of its own start times; unbounded DFS equals the
exhaustive optimum on small plans, and no algorithm beats it; the lower
bound is the definition's; the naive and load-balance-only schedules are
the ones their definitions fix; the ensemble is the better of its two
searches; the randomized search reaches the lower bound on Table 3 (Section
5.3.1).  Budget-limited DFS and the randomized search's exact schedule have
several correct answers: they are checked by these properties only.
"""

import itertools
import json
import math
import os
import random
import zlib

import pytest

import oracle
from oracle import schedule as S
from paper_2211_05322_amd import binding as B
from paper_2211_05322_amd.workloads import WORKLOADS
from tests.test_capi_host import _fuzz

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
ALGOS = ["naive", "load_balance", "dfs", "randomized", "ensemble"]


def _table3():
    with open(os.path.join(GOLDEN, "table3_cases.json")) as f:
        return json.load(f)


def random_model(rng, n, nsrc_hosts, ndst_hosts):
    model = []
    for _ in range(n):
        dur = rng.choice([1, 2, 3, 5, 8])
        cand = sorted(rng.sample(range(nsrc_hosts), rng.randint(1, nsrc_hosts)))
        recv = sorted(rng.sample(range(nsrc_hosts, nsrc_hosts + ndst_hosts), rng.randint(1, ndst_hosts)))
        model.append((dur, cand, recv))
    return model, nsrc_hosts + ndst_hosts


# ------------------------------------------------------------ oracle pins

@pytest.mark.parametrize("seed", range(40))
def test_oracle_against_exhaustive_search(seed):
    rng = random.Random(seed)
    model, nh = random_model(rng, rng.randint(1, 5), rng.randint(1, 3), rng.randint(1, 3))
    opt = S.optimum(model, nh)
    assert S.lower_bound(model, nh) <= opt
    full = S.dfs(model, nh, 10**9)
    assert full["makespan"] == opt, "unbounded DFS must find the optimum"
    for sched in (S.naive(model, nh), S.load_balance(model, nh), full, S.randomized(model, nh, 8, seed),
                  S.ensemble(model, nh, 50, 8, seed), S.dfs(model, nh, 3)):
        assert S.valid(model, sched)
        assert sched["makespan"] >= opt
        assert sched["makespan"] == S.completion_time(model, sched)


@pytest.mark.parametrize("seed", range(4))
def test_dfs_reaches_exhaustive_optimum_on_larger_sets(seed):
    # 7 tasks with their sender host fixed: the optimum is the best of the
    # 7! orders; 5 tasks with two candidate senders each: 5! x 2^5 schedules
    rng = random.Random(100 + seed)
    for n, ncand in ((7, 1), (5, 2)):
        model = []
        for _ in range(n):
            cand = sorted(rng.sample(range(3), ncand))
            recv = sorted(rng.sample(range(3, 6), rng.randint(1, 2)))
            model.append((rng.choice([1, 2, 3, 5]), cand, recv))
        opt = S.optimum(model, 6)
        full = S.dfs(model, 6, 10**9)
        assert full["makespan"] == opt and S.valid(model, full)
        assert S.lower_bound(model, 6) <= opt
        for sched in (S.naive(model, 6), S.load_balance(model, 6), S.randomized(model, 6, 8, seed)):
            assert S.valid(model, sched) and sched["makespan"] >= opt


def test_start_times_by_hand():
    # hosts 0, 1 send, 2, 3 receive.  A: 0 -> {2}, 3 long; B: 1 -> {2}, 2
    # long; C: 1 -> {3}, 1 long.  Order A, B, C: B waits for A on host 2
    # (starts 3), C for B on host 1 (starts 5), makespan 6.  Order C, A, B:
    # C and A start at 0, B waits for C (host 1, ends 1) and A (host 2,
    # ends 3): starts 3, makespan 5.
    model = [(3, [0], [2]), (2, [1], [2]), (1, [1], [3])]
    host = [0, 1, 1]
    assert S.start_times(model, [0, 1, 2], host) == [0, 3, 5]
    assert S.schedule(model, [0, 1, 2], host)["makespan"] == 6
    assert S.start_times(model, [2, 0, 1], host) == [0, 3, 0]
    assert S.schedule(model, [2, 0, 1], host)["makespan"] == 5
    assert S.optimum(model, 4) == 5


def test_valid_is_eq2_and_eq3():
    model = [(3, [0], [2]), (2, [1], [2]), (1, [0, 1], [3])]
    ok = {"host": [0, 1, 1], "start": [0, 3, 0]}
    assert S.valid(model, ok)
    # B overlaps A on receiver host 2
    assert not S.valid(model, {"host": [0, 1, 1], "start": [0, 2, 0]})
    # C on the sender host of A while A runs
    assert not S.valid(model, {"host": [0, 1, 0], "start": [0, 3, 1]})
    # back to back is not an overlap (open intervals)
    assert S.valid(model, {"host": [0, 1, 0], "start": [0, 3, 3]})
    # Eq. 2: host 1 holds no replica of A
    assert not S.valid(model, {"host": [1, 1, 1], "start": [0, 3, 5]})


def test_lower_bound_is_tight_when_one_host_carries_everything():
    model = [(3, [0], [2]), (4, [1], [2]), (5, [0, 1], [2])]
    assert S.lower_bound(model, 3) == 12 == S.optimum(model, 3)


def test_load_balance_visits_longest_first():
    # Eq. 4 greedy, by hand: durations 1, 1, 2, each sendable from hosts 0
    # or 1, each to its own receiver.  Longest first: the 2 goes to host 0,
    # then both 1s to host 1 -> loads 2 and 2, makespan 2.  Shortest first
    # would give host 0 a 1 and the 2 -> makespan 3.
    model = [(1, [0, 1], [2]), (1, [0, 1], [3]), (2, [0, 1], [4])]
    sched = S.load_balance(model, 5)
    assert sched["host"] == [1, 1, 0] and sched["makespan"] == 2 and S.valid(model, sched)


@pytest.mark.parametrize("n,hosts", [(4, 2), (6, 3), (7, 2), (5, 4)])
def test_load_balance_is_eq4_optimal_for_equal_durations(n, hosts):
    # equal durations, every task sendable from every host: the greedy deals
    # them round robin, ceil(n / hosts) each, which the exhaustive Eq. 4
    # minimum confirms
    model = [(3, list(range(hosts)), [hosts + i]) for i in range(n)]
    nh = hosts + n
    sched = S.load_balance(model, nh)
    load = [0] * nh
    for h, m in zip(sched["host"], model):
        load[h] += m[0]
    assert max(load) == 3 * math.ceil(n / hosts) == S.optimum_sender_load(model, nh)


def test_randomized_depends_only_on_seed():
    rng = random.Random(3)
    model, nh = random_model(rng, 6, 3, 3)
    assert S.randomized(model, nh, 4, 11) == S.randomized(model, nh, 4, 11)


def test_randomized_starts_disjoint_tasks_together_and_serialises_conflicts():
    # four tasks on disjoint hosts all start at 0; four tasks into one
    # receiver run one after another
    disjoint = [(2, [i], [4 + i]) for i in range(4)]
    sched = S.randomized(disjoint, 8, 4, 0)
    assert sched["start"] == [0, 0, 0, 0] and sched["makespan"] == 2
    shared = [(d, [i], [4]) for i, d in enumerate((1, 2, 3, 4))]
    sched = S.randomized(shared, 5, 4, 0)
    assert S.valid(shared, sched) and sched["makespan"] == 10


def test_randomized_search_over_orders_finds_the_larger_set():
    # hosts 0-2 send, 3-5 receive.  A: 3 long, 0 -> {5}; B: 2 long, 1 or 2 ->
    # {4, 5}; C: 2 long, 0 or 1 -> {3}; D: 3 long, 0 or 1 -> {4}.  Hosts 4
    # and 5 each need 5 units of work, so 5 is the bound, and it is reached
    # (A and D at 0, then B and C at 3).  A single order that starts with D
    # on host 0 picks {D, C} (4 hosts) and leaves A and B to collide on host
    # 5 later; searching several orders for the set with the most hosts
    # starts {B, C} (5 hosts) and reaches 5.
    model = [(3, [0], [5]), (2, [1, 2], [4, 5]), (2, [0, 1], [3]), (3, [0, 1], [4])]
    assert S.lower_bound(model, 6) == S.optimum(model, 6) == 5
    for seed in range(10):
        sched = S.randomized(model, 6, 16, seed)
        assert S.valid(model, sched) and sched["makespan"] == 5, seed


# ---------------------------------------------------- the paper's cases

def _case_model(c, shape=None):
    g = _table3()
    shape = tuple(shape or g["tensor_shape"])
    sm, dm = tuple(c["send_mesh"]), tuple(c["recv_mesh"])
    # a node is a mesh row (Section 5.1.2: 2-node meshes of 4 GPUs)
    return S.build_model(shape, 2, sm, c["send_spec"], dm, c["recv_spec"], sm[-1], dm[-1])


def test_table3_case2_naive_congests_first_node():
    # Section 5.3.1: in case 2 the naive algorithm sends all tensors from
    # the first node; balancing the two senders halves the time
    c = _table3()["cases"][1]
    tasks, model, nh = _case_model(c)
    nv = S.naive(model, nh)
    assert {h for h in nv["host"]} == {0}
    assert nv["makespan"] == 2 * S.lower_bound(model, nh) == 2 * S.load_balance(model, nh)["makespan"]


def test_table3_case8_single_broadcast():
    c = _table3()["cases"][7]
    tasks, model, nh = _case_model(c)
    assert len(model) == 1


def test_table3_ordering_reaches_lower_bound():
    # Section 5.3.1: the ordered schedule keeps no send or receive node idle;
    # "load balance only" congests in the cases with replicated senders or
    # more tasks than nodes (3, 5, 6, 9)
    for c in _table3()["cases"]:
        tasks, model, nh = _case_model(c)
        lb = S.lower_bound(model, nh)
        assert S.randomized(model, nh, 16, 0)["makespan"] == lb, c["case"]
        if len(model) <= 4:
            assert S.optimum(model, nh) == lb
        if c["case"] in (3, 5, 6, 9):
            assert S.load_balance(model, nh)["makespan"] > lb, c["case"]


# ------------------------------------------------- the library's scheduler

def _library(plan, model, tasks, sph, dph, algo, budget, rounds, seed):
    got = B.reshard_schedule(plan, sph, dph, algo, max_dfs_nodes=budget, random_rounds=rounds, seed=seed)
    for i, d in enumerate(got["senders"]):
        assert d in tasks[i]["senders"], (algo, i)
    return got, {"host": [d // sph for d in got["senders"]], "start": got["starts"], "makespan": got["makespan"]}


def check_library(shape, dtype, sm, ss, dm, ds, sph, dph, budget=3000, rounds=6, seed=5, exact=False):
    """Every algorithm of the library on one plan, against facts only."""
    import numpy as np
    es = np.dtype(dtype).itemsize
    p = B.reshard_plan(shape, dtype, sm, ss, dm, ds)
    tasks, model, nh = S.build_model(shape, es, sm, ss, dm, ds, sph, dph)
    lb = S.lower_bound(model, nh)
    opt = S.optimum(model, nh) if exact else None
    out = {}
    for algo in ALGOS:
        got, sched = _library(p, model, tasks, sph, dph, algo, budget, rounds, seed)
        assert S.valid(model, sched), algo
        assert got["makespan"] == S.completion_time(model, sched), algo
        assert got["lower_bound"] == lb, algo
        assert got["makespan"] >= (opt if exact else lb), algo
        out[algo] = (got, sched)
    # naive: the lowest-indexed owner sends, tasks in unit-task order
    got, sched = out["naive"]
    assert got["senders"] == oracle.choose_senders_naive(tasks)
    assert sched["start"] == S.naive(model, nh)["start"]
    # load balance only: Eq. 4's greedy with the stated ties
    want = S.load_balance(model, nh)
    assert out["load_balance"][1]["host"] == want["host"] and out["load_balance"][0]["starts"] == want["start"]
    # the search starts from the load-balance schedule; the ensemble keeps
    # the better of its two searches
    assert out["dfs"][0]["makespan"] <= want["makespan"]
    assert out["ensemble"][0]["makespan"] == min(out["dfs"][0]["makespan"], out["randomized"][0]["makespan"])
    if exact:
        full, _ = _library(p, model, tasks, sph, dph, "dfs", 10**8, rounds, seed)
        assert full["makespan"] == opt, "unbounded DFS must find the optimum"
    return out, lb


def _small_enough(model):
    n = len(model)
    return n <= 6 and math.prod(len(m[1]) for m in model) * math.factorial(n) <= 20000


@pytest.mark.parametrize("case", range(1, 10))
def test_library_table3(case):
    c = _table3()["cases"][case - 1]
    sm, dm = tuple(c["send_mesh"]), tuple(c["recv_mesh"])
    check_library((64, 48, 40), "float16", sm, c["send_spec"], dm, c["recv_spec"], sm[-1], dm[-1])


def test_library_table3_full_size_reaches_bound():
    # Section 5.3.1, at the paper's tensor: the ordered schedule keeps every
    # node busy, i.e. reaches the lower bound, in all nine cases
    g = _table3()
    for c in g["cases"]:
        sm, dm = tuple(c["send_mesh"]), tuple(c["recv_mesh"])
        shape = tuple(g["tensor_shape"])
        p = B.reshard_plan(shape, "float16", sm, c["send_spec"], dm, c["recv_spec"])
        tasks, model, nh = _case_model(c)
        for algo in ("randomized", "ensemble"):
            got, sched = _library(p, model, tasks, sm[-1], dm[-1], algo, 2000, 16, 0)
            assert S.valid(model, sched) and got["makespan"] == S.completion_time(model, sched)
            assert got["makespan"] == got["lower_bound"] == S.lower_bound(model, nh), (c["case"], algo)


@pytest.mark.parametrize("wid", sorted(WORKLOADS))
def test_library_workloads(wid):
    w = WORKLOADS[wid]
    small = {1: (64, 96), 2: (4, 64, 96), 3: (2, 24, 200), 4: (4, 8, 66, 16), 5: (2, 64, 384)}[wid]
    check_library(small, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec, w.src_mesh[-1],
                  w.dst_mesh[-1], budget=500)


def _fuzz_plans(n, seed):
    out = []
    for case in _fuzz(n, seed):
        shape, dt, sm, ss, dm, ds, _ = case
        rng = random.Random(zlib.crc32(repr(case).encode()))
        sph = rng.randint(1, math.prod(sm))
        dph = rng.randint(1, math.prod(dm))
        out.append((shape, dt, sm, ss, dm, ds, sph, dph))
    return out


@pytest.mark.parametrize("case", _fuzz_plans(30, 77))
def test_library_fuzz(case):
    shape, dt, sm, ss, dm, ds, sph, dph = case
    import numpy as np
    _, model, _ = S.build_model(shape, np.dtype(dt).itemsize, sm, ss, dm, ds, sph, dph)
    check_library(shape, dt, sm, ss, dm, ds, sph, dph, budget=400, exact=_small_enough(model))


def test_library_exact_on_small_plans():
    # plans small enough for the exhaustive optimum: unbounded DFS reaches
    # it and nothing beats it
    import numpy as np
    checked = 0
    for case in _fuzz_plans(400, 1234):
        shape, dt, sm, ss, dm, ds, sph, dph = case
        _, model, _ = S.build_model(shape, np.dtype(dt).itemsize, sm, ss, dm, ds, sph, dph)
        if len(model) < 2 or not _small_enough(model):
            continue
        check_library(shape, dt, sm, ss, dm, ds, sph, dph, budget=200, exact=True)
        checked += 1
        if checked == 40:
            break
    assert checked >= 20


def test_schedule_errors():
    p = B.reshard_plan((4, 4), "float16", (2,), "S^0R", (2,), "RS^0")
    for bad in ({"src_devices_per_host": 0}, {"max_dfs_nodes": -1}):
        kw = {"src_devices_per_host": 1, "dst_devices_per_host": 1, **bad}
        with pytest.raises(B.ReshardError):
            B.reshard_schedule(p, kw["src_devices_per_host"], kw["dst_devices_per_host"],
                               max_dfs_nodes=kw.get("max_dfs_nodes", 10))


def test_workload_table3_matches_golden():
    from paper_2211_05322_amd.workloads import TABLE3_CASES, TABLE3_SHAPE
    g = _table3()
    assert tuple(g["tensor_shape"]) == TABLE3_SHAPE
    for (case, ss, ds, sm, dm), c in zip(TABLE3_CASES, g["cases"]):
        assert case == c["case"] and sm == tuple(c["send_mesh"]) and dm == tuple(c["recv_mesh"])
        assert oracle.parse_spec(ss, 3, len(sm)) == oracle.parse_spec(c["send_spec"], 3, len(sm))
        assert oracle.parse_spec(ds, 3, len(dm)) == oracle.parse_spec(c["recv_spec"], 3, len(dm))


def test_exhaustive_helpers_agree_on_a_tiny_case():
    # optimum over (assignment x order) equals a direct search over start
    # times on an integer grid for two tasks sharing a receiver
    model = [(2, [0, 1], [2]), (3, [0], [2])]
    best = min(max(s0 + 2, s1 + 3)
               for h0 in (0, 1) for s0, s1 in itertools.product(range(6), range(6))
               if S.valid(model, {"host": [h0, 0], "start": [s0, s1]}))
    assert S.optimum(model, 3) == best == 5
