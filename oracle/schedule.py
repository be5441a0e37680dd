"""Oracle for the unit-task scheduling of Section 3.2 -- test infrastructure.

Only the test suite may import this module; the library never does.

The cluster model of Section 3.2 (Eq. 1-3): unit task i has a duration T_i,
the hosts n_i holding a replica of its slice (candidate senders) and the
receiver hosts m_i.  A schedule picks one sender host n_i* in n_i (Eq. 2)
and a start time S_i; two tasks that share the sender host or any receiver
host must not run at the same time (Eq. 3); the objective is the completion
time of the last task, max_i S_i + T_i (Eq. 1).

Readings (the paper leaves these open):
* hosts: device d of a mesh is on host d // devices_per_host; destination
  hosts are numbered after the source hosts (the two meshes are disjoint);
* T_i is the slice's byte count: a broadcast costs about one transfer of
  the slice whatever the number of receivers (Section 3.1);
* start times follow the paper's reduction to per-host orders: given a
  global order, a task starts as soon as every earlier task that uses one of
  its hosts has finished;
* naive: the lowest-indexed owner device sends; tasks run in unit-task order;
* load balance only: Eq. 4's greedy -- longest task first (equal durations
  keep the unit-task order), each to the candidate host with the least load
  so far (equal loads: the lowest host index); the tasks then run in that
  greedy order (Section 5.3.1);
* DFS with pruning: the search tree branches on the next task of the global
  order together with its sender host; a branch is cut when its lower bound
  -- per host, the finish time of the tasks placed so far plus the durations
  of the unplaced tasks that must use that host -- is not below the best
  completion time found so far (a tie cannot improve on it); the budget is
  a count of tree nodes, and the search always completes its first descent,
  so it returns a schedule under any budget;
* greedy search with randomization: one iteration per point in time at
  which a host becomes free; among the unscheduled tasks whose receiver
  hosts are all idle and which have an idle candidate host, several random
  orders (Python's Mersenne Twister, seeded) each pick tasks greedily in
  their order; a picked task takes its idle candidate host with the least
  bytes sent so far (equal: lowest index); the order whose set involves the
  most hosts is started (equal: the first drawn);
* ensemble: the better of DFS and the randomized search (equal: DFS).

The exact optimum: an optimal schedule's tasks, sorted by start time and
rescheduled by the reduction above, start no later, so the minimum over
every sender assignment and every global order is the optimum of Eq. 1-3
(brute force, for a handful of tasks).

Pinned by that brute force, by the definition of validity (Eq. 2-3) and by
the statements of Section 5.3.1 on the Table 3 cases (tests/test_schedule.py).
"""

import itertools
import random

from .reshard import parse_spec, unit_tasks


def build_model(shape, itemsize, src_mesh, src_spec, dst_mesh, dst_spec, src_per_host, dst_per_host):
    """Unit tasks -> (tasks, [(T_i, candidate sender hosts n_i, receiver hosts m_i)], number of hosts)."""
    tasks = unit_tasks(shape, src_mesh, src_spec, dst_mesh, dst_spec)
    n_src = 1
    for m in src_mesh:
        n_src *= m
    n_dst = 1
    for m in dst_mesh:
        n_dst *= m
    src_hosts = -(-n_src // src_per_host)
    dst_hosts = -(-n_dst // dst_per_host)
    model = []
    for t in tasks:
        volume = 1
        for lo, hi in t["box"]:
            volume *= hi - lo
        senders = sorted(set(d // src_per_host for d in t["senders"]))
        receivers = sorted(set(src_hosts + d // dst_per_host for d in t["receivers"]))
        model.append((volume * itemsize, senders, receivers))
    return tasks, model, src_hosts + dst_hosts


def _hosts_of(model, i, host):
    return {host[i], *model[i][2]}


def start_times(model, order, host):
    """The paper's reduction: task i starts when every task before it in
    `order` that shares one of its hosts (sender or receivers) has finished."""
    start = [None] * len(model)
    for pos, i in enumerate(order):
        mine = _hosts_of(model, i, host)
        s = 0
        for j in order[:pos]:
            if mine & _hosts_of(model, j, host):
                s = max(s, start[j] + model[j][0])
        start[i] = s
    return start


def schedule(model, order, host):
    start = start_times(model, list(order), host)
    return {"host": list(host), "start": start, "makespan": max((s + m[0] for s, m in zip(start, model)), default=0)}


def list_schedule(model, order, host, nhosts):
    """Start times of a global order and sender hosts (kept for callers that pass a host count)."""
    return schedule(model, order, host)


def completion_time(model, sched):
    """Eq. 1: the end of the last task."""
    return max((s + m[0] for s, m in zip(sched["start"], model)), default=0)


def valid(model, sched):
    """Eq. 2 (each sender holds the slice) and Eq. 3 (tasks sharing the
    sender host or a receiver host do not overlap in time)."""
    n = len(model)
    for i in range(n):
        if sched["host"][i] not in model[i][1] or sched["start"][i] < 0:
            return False
    for i in range(n):
        for j in range(i + 1, n):
            share = sched["host"][i] == sched["host"][j] or set(model[i][2]) & set(model[j][2])
            if not share:
                continue
            a0, a1 = sched["start"][i], sched["start"][i] + model[i][0]
            b0, b1 = sched["start"][j], sched["start"][j] + model[j][0]
            if max(a0, b0) < min(a1, b1):
                return False
    return True


def required_work(model, nhosts, tasks=None):
    """Per host: the durations of the tasks (all, or those listed) that must
    use it -- every receiver host, and the sender host when only one host
    holds the slice."""
    work = [0] * nhosts
    for i in range(len(model)) if tasks is None else tasks:
        dur, senders, receivers = model[i]
        involved = set(receivers) | (set(senders) if len(senders) == 1 else set())
        for h in involved:
            work[h] += dur
    return work


def lower_bound(model, nhosts):
    """No schedule ends before the busiest host's required work, nor before
    the longest task (the Eq. 4 style bound of Section 3.2)."""
    return max([0] + required_work(model, nhosts) + [m[0] for m in model])


def naive(model, nhosts):
    return schedule(model, range(len(model)), [m[1][0] for m in model])


def load_balance(model, nhosts):
    order = sorted(range(len(model)), key=lambda i: -model[i][0])  # stable: ties keep task order
    sent = [0] * nhosts
    host = [None] * len(model)
    for i in order:
        h = min(model[i][1], key=lambda c: (sent[c], c))
        host[i] = h
        sent[h] += model[i][0]
    return schedule(model, order, host)


def dfs(model, nhosts, budget):
    """Depth-first search over (next task, its sender host) with pruning."""
    n = len(model)
    best = {"sched": None, "span": float("inf")}
    nodes = [0]

    def bound(order, host):
        start = start_times(model, order, host)
        finish = [0] * nhosts
        for i in order:
            for h in _hosts_of(model, i, host):
                finish[h] = max(finish[h], start[i] + model[i][0])
        rest = required_work(model, nhosts, [i for i in range(n) if i not in order])
        return max([0] + [f + r for f, r in zip(finish, rest)])

    def visit(order, host):
        if len(order) == n:
            sched = schedule(model, order, host)
            if sched["makespan"] < best["span"]:
                best["sched"], best["span"] = sched, sched["makespan"]
            return
        for i in range(n):
            if i in order:
                continue
            for h in model[i][1]:
                if best["sched"] is not None and nodes[0] >= budget:
                    return
                nodes[0] += 1
                host[i] = h
                order.append(i)
                if bound(order, host) < best["span"]:
                    visit(order, host)
                order.pop()
                host[i] = None

    visit([], [None] * n)
    out = dict(best["sched"]) if best["sched"] is not None else schedule(model, [], [])
    out["nodes"] = nodes[0]
    return out


def randomized(model, nhosts, rounds, seed):
    """Greedy search with randomization (Section 3.2)."""
    n = len(model)
    rng = random.Random(seed)
    host, start = [None] * n, [None] * n
    busy_until = [0] * nhosts
    sent = [0] * nhosts
    todo = list(range(n))
    now = 0
    while todo:
        idle = {h for h in range(nhosts) if busy_until[h] <= now}
        best_set, best_hosts = [], -1
        for _ in range(max(1, rounds)):
            order = list(todo)
            rng.shuffle(order)
            free = set(idle)
            picked = []
            for i in order:
                dur, senders, receivers = model[i]
                if not set(receivers) <= free:
                    continue
                usable = [c for c in senders if c in free]
                if not usable:
                    continue
                h = min(usable, key=lambda c: (sent[c], c))
                free -= {h, *receivers}
                picked.append((i, h))
            involved = sum(1 + len(model[i][2]) for i, _ in picked)
            if involved > best_hosts:
                best_set, best_hosts = picked, involved
        for i, h in best_set:
            host[i], start[i] = h, now
            sent[h] += model[i][0]
            for q in {h, *model[i][2]}:
                busy_until[q] = now + model[i][0]
        done = {i for i, _ in best_set}
        todo = [i for i in todo if i not in done]
        later = [b for b in busy_until if b > now]
        if todo and later:
            now = min(later)
    return {"host": host, "start": start, "makespan": max((s + m[0] for s, m in zip(start, model)), default=0)}


def ensemble(model, nhosts, budget, rounds, seed):
    a = dfs(model, nhosts, budget)
    b = randomized(model, nhosts, rounds, seed)
    return b if b["makespan"] < a["makespan"] else a


def optimum(model, nhosts):
    """Exact minimum of Eq. 1 subject to Eq. 2-3: every sender assignment x
    every global order."""
    best = None
    for host in itertools.product(*[m[1] for m in model]):
        for order in itertools.permutations(range(len(model))):
            span = schedule(model, order, list(host))["makespan"]
            if best is None or span < best:
                best = span
    return best if best is not None else 0


def optimum_sender_load(model, nhosts):
    """Exact minimum of Eq. 4: the busiest sender host's total duration over
    every sender assignment."""
    best = None
    for host in itertools.product(*[m[1] for m in model]):
        load = [0] * nhosts
        for h, m in zip(host, model):
            load[h] += m[0]
        if best is None or max(load) < best:
            best = max(load)
    return best if best is not None else 0


def sender_devices(tasks, sched, src_per_host):
    """Sender device per task: its lowest-indexed owner on the chosen host."""
    return [min(d for d in t["senders"] if d // src_per_host == h) for t, h in zip(tasks, sched["host"])]


__all__ = ["build_model", "start_times", "schedule", "list_schedule", "completion_time", "valid",
           "required_work", "lower_bound", "naive", "load_balance", "dfs", "randomized", "ensemble", "optimum",
           "optimum_sender_load", "sender_devices", "parse_spec"]
