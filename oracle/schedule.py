"""Oracle for the unit-task scheduling of Section 3.2 -- test infrastructure.

The cluster model of Section 3 and Eq. 1-3: each unit task i has a duration
T_i, candidate sender hosts n_i (hosts holding a replica of its slice) and
receiver hosts m_i.  A schedule picks a sender host n_i* in n_i and a start
time S_i such that tasks sharing the sender host or any receiver host do not
overlap; the objective is the makespan max_i S_i + T_i.  Hosts: device d of a
mesh is on host d // devices_per_host; destination hosts are numbered after
the source hosts (the meshes are disjoint).  T_i is the slice's byte count:
a broadcast costs about one transfer of the slice whatever the receiver
count (Section 3.1).

Start times follow the paper's reduction: given a global order and the
sender hosts, each task starts when every earlier task on its hosts has
finished.  The exact optimum is attained by such a list schedule (order the
tasks of an optimal schedule by start time; none starts later), so the
brute force below enumerates sender assignments and orders.

The algorithms are written out from Section 3.2 with the tie-breaking the
library uses, so their results can be compared exactly:
* naive: lowest-indexed owner's host, task order;
* load balance only (Eq. 4): longest first to the least-loaded candidate
  host, run in that order;
* DFS with pruning: branch on (next task, sender host); prune when the
  per-host bound (host free time + work certain to land on it) is not below
  the best makespan; identical tasks are branched on once; a branch budget
  stands in for the time budget;
* greedy search with randomization: from the current time, draw random
  orders of the unscheduled tasks (SplitMix64, Steele et al. 2014, Fisher-
  Yates), take every task whose receivers and some candidate sender host are
  idle, keep the order whose set busies the most hosts, start it, advance to
  the next finish;
* ensemble: the better of DFS and randomized (ties: DFS).

Pinned by exhaustive search (tests/test_schedule.py).
"""

import itertools

from .reshard import parse_spec, unit_tasks

MASK64 = (1 << 64) - 1


def build_model(shape, itemsize, src_mesh, src_spec, dst_mesh, dst_spec, src_per_host, dst_per_host):
    """Unit tasks -> list of (duration, candidate sender hosts, receiver hosts)."""
    tasks = unit_tasks(shape, src_mesh, src_spec, dst_mesh, dst_spec)
    n_src = 1
    for m in src_mesh:
        n_src *= m
    hs = (n_src + src_per_host - 1) // src_per_host
    model = []
    for t in tasks:
        vol = 1
        for lo, hi in t["box"]:
            vol *= hi - lo
        cand = sorted({d // src_per_host for d in t["senders"]})
        recv = sorted({hs + d // dst_per_host for d in t["receivers"]})
        model.append((vol * itemsize, cand, recv))
    n_dst = 1
    for m in dst_mesh:
        n_dst *= m
    nhosts = hs + (n_dst + dst_per_host - 1) // dst_per_host
    return tasks, model, nhosts


def list_schedule(model, order, host, nhosts):
    free = [0] * nhosts
    start = [0] * len(model)
    span = 0
    for i in order:
        dur, _, recv = model[i]
        s = max([free[host[i]]] + [free[r] for r in recv])
        for h in [host[i]] + list(recv):
            free[h] = s + dur
        start[i] = s
        span = max(span, s + dur)
    return {"host": list(host), "start": start, "makespan": span}


def lower_bound(model, nhosts):
    must = [0] * nhosts
    lb = 0
    for dur, cand, recv in model:
        for r in recv:
            must[r] += dur
        if len(cand) == 1:
            must[cand[0]] += dur
        lb = max(lb, dur)
    return max([lb] + must)


def valid(model, sched):
    """Every task on a candidate host; tasks sharing a host never overlap."""
    ivs = {}
    for i, (dur, cand, recv) in enumerate(model):
        if sched["host"][i] not in cand:
            return False
        for h in [sched["host"][i]] + list(recv):
            ivs.setdefault(h, []).append((sched["start"][i], sched["start"][i] + dur))
    for v in ivs.values():
        v.sort()
        for (a0, a1), (b0, b1) in zip(v, v[1:]):
            if b0 < a1:
                return False
    return True


def naive(model, nhosts):
    return list_schedule(model, range(len(model)), [c[0] for _, c, _ in model], nhosts)


def load_balance(model, nhosts):
    order = sorted(range(len(model)), key=lambda i: (-model[i][0], i))
    load = [0] * nhosts
    host = [None] * len(model)
    for i in order:
        best = min(model[i][1], key=lambda h: (load[h], h))
        host[i] = best
        load[best] += model[i][0]
    return list_schedule(model, order, host, nhosts)


def dfs(model, nhosts, max_nodes):
    n = len(model)
    cls = []
    for i in range(n):
        c = i
        for j in range(i):
            if model[j] == model[i]:
                c = cls[j]
                break
        cls.append(c)
    must = [0] * nhosts
    for dur, cand, recv in model:
        for r in recv:
            must[r] += dur
        if len(cand) == 1:
            must[cand[0]] += dur
    best = load_balance(model, nhosts)
    state = {"nodes": 0, "best": best}
    free = [0] * nhosts
    done = [False] * n
    order, host = [], [None] * n

    def go(span):
        if len(order) == n:
            if span < state["best"]["makespan"]:
                state["best"] = list_schedule(model, order, host, nhosts)
            return
        seen = set()
        for i in range(n):
            if done[i] or cls[i] in seen:
                continue
            seen.add(cls[i])
            dur, cand, recv = model[i]
            for h in cand:
                if state["nodes"] >= max_nodes:
                    return
                state["nodes"] += 1
                s = max([free[h]] + [free[r] for r in recv])
                fin = s + dur
                saved = {q: free[q] for q in [h] + list(recv)}
                for q in [h] + list(recv):
                    free[q] = fin
                for r in recv:
                    must[r] -= dur
                if len(cand) == 1:
                    must[h] -= dur
                lb = max([span, fin] + [free[q] + must[q] for q in range(nhosts)])
                if lb < state["best"]["makespan"]:
                    done[i] = True
                    order.append(i)
                    host[i] = h
                    go(max(span, fin))
                    order.pop()
                    done[i] = False
                if len(cand) == 1:
                    must[h] += dur
                for r in recv:
                    must[r] += dur
                for q in reversed([h] + list(recv)):
                    free[q] = saved[q]
        return

    go(0)
    out = dict(state["best"])
    out["nodes"] = state["nodes"]
    return out


def splitmix64(state):
    """One SplitMix64 step: returns (new state, output)."""
    state = (state + 0x9E3779B97F4A7C15) & MASK64
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return state, z ^ (z >> 31)


def randomized(model, nhosts, rounds, seed):
    n = len(model)
    host = [None] * n
    start = [0] * n
    span = 0
    rng = seed & MASK64
    remaining = list(range(n))
    busy = [0] * nhosts
    now = 0
    while remaining:
        best_set, best_score = [], -1
        for _ in range(max(1, rounds)):
            perm = list(remaining)
            for i in range(len(perm), 1, -1):
                rng, z = splitmix64(rng)
                j = z % i
                perm[i - 1], perm[j] = perm[j], perm[i - 1]
            used = [b > now for b in busy]
            chosen, score = [], 0
            for i in perm:
                dur, cand, recv = model[i]
                if any(used[r] for r in recv):
                    continue
                free_c = [c for c in cand if not used[c]]
                if not free_c:
                    continue
                h = free_c[0]
                used[h] = True
                for r in recv:
                    used[r] = True
                chosen.append((i, h))
                score += 1 + len(recv)
            if score > best_score:
                best_set, best_score = chosen, score
        for i, h in best_set:
            host[i] = h
            start[i] = now
            fin = now + model[i][0]
            busy[h] = fin
            for r in model[i][2]:
                busy[r] = fin
            span = max(span, fin)
        picked = {i for i, _ in best_set}
        remaining = [i for i in remaining if i not in picked]
        if not remaining:
            break
        later = [b for b in busy if b > now]
        if later:
            now = min(later)
    return {"host": host, "start": start, "makespan": span}


def ensemble(model, nhosts, max_nodes, rounds, seed):
    a = dfs(model, nhosts, max_nodes)
    b = randomized(model, nhosts, rounds, seed)
    return b if b["makespan"] < a["makespan"] else a


def optimum(model, nhosts):
    """Exact minimum makespan: every sender assignment x every order."""
    best = None
    n = len(model)
    for host in itertools.product(*[cand for _, cand, _ in model]):
        for order in itertools.permutations(range(n)):
            m = list_schedule(model, order, host, nhosts)["makespan"]
            if best is None or m < best:
                best = m
    return best


def sender_devices(tasks, sched, src_per_host):
    """Sender device per task: its lowest-indexed owner on the chosen host."""
    return [min(d for d in t["senders"] if d // src_per_host == h) for t, h in zip(tasks, sched["host"])]


__all__ = ["build_model", "list_schedule", "lower_bound", "valid", "naive", "load_balance", "dfs",
           "randomized", "ensemble", "optimum", "sender_devices", "parse_spec"]
