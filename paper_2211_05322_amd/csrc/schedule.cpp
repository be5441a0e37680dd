// schedule.cpp -- sender choice and ordering of unit tasks under the paper's
// cluster model (Section 3.2, Eq. 1-3): every task occupies its sender host
// and all its receiver hosts for its whole duration; two tasks that share a
// host may not overlap.  Minimise the makespan.
//
// Hosts: device d of a mesh lives on host d / devices_per_host; source and
// destination meshes are disjoint, so destination hosts are numbered after
// the source hosts.  A task's duration is its slice's byte count (a broadcast
// costs about one transfer of the slice regardless of the receiver count,
// Section 3.1).  A schedule is a global order plus a sender host per task;
// each task starts when every earlier task on its hosts has finished (the
// paper's reduction of the start times to per-host orders).
#include <algorithm>
#include <cstdint>
#include <set>
#include <string>
#include <vector>

#include "../../include/reshard.h"
#include "planner.hpp"
#include "status.hpp"

namespace rs {

namespace {

struct STask {
    int64_t dur = 0;
    std::vector<int32_t> cand;  // candidate sender hosts, ascending, distinct
    std::vector<int32_t> recv;  // receiver hosts, ascending, distinct
};

struct Sched {
    std::vector<int32_t> host;   // chosen sender host per task
    std::vector<int64_t> start;  // start time per task
    int64_t makespan = 0;
};

// SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number
// generators", OOPSLA 2014).
struct SplitMix64 {
    uint64_t x;
    uint64_t next() {
        uint64_t z = (x += 0x9E3779B97F4A7C15ull);
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
};

// List schedule of a global order with given sender hosts.
Sched list_schedule(const std::vector<STask> &ts, const std::vector<int32_t> &order,
                    const std::vector<int32_t> &host, int nhosts) {
    Sched s;
    s.host = host;
    s.start.assign(ts.size(), 0);
    std::vector<int64_t> free_at(nhosts, 0);
    for (int32_t i : order) {
        int64_t st = free_at[host[i]];
        for (int32_t r : ts[i].recv) st = std::max(st, free_at[r]);
        const int64_t fin = st + ts[i].dur;
        free_at[host[i]] = fin;
        for (int32_t r : ts[i].recv) free_at[r] = fin;
        s.start[i] = st;
        s.makespan = std::max(s.makespan, fin);
    }
    return s;
}

// Naive algorithm: the owner with the lowest device index sends; tasks run
// in task order.
Sched naive(const std::vector<STask> &ts, int nhosts) {
    std::vector<int32_t> order(ts.size()), host(ts.size());
    for (size_t i = 0; i < ts.size(); ++i) {
        order[i] = int32_t(i);
        host[i] = ts[i].cand.front();
    }
    return list_schedule(ts, order, host, nhosts);
}

// Load balance only (Eq. 4): longest first, each task to the candidate host
// with the least load so far (ties: lowest host); that greedy order is also
// the execution order.
Sched load_balance(const std::vector<STask> &ts, int nhosts) {
    std::vector<int32_t> order(ts.size()), host(ts.size());
    for (size_t i = 0; i < ts.size(); ++i) order[i] = int32_t(i);
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return ts[a].dur > ts[b].dur; });
    std::vector<int64_t> load(nhosts, 0);
    for (int32_t i : order) {
        int32_t best = ts[i].cand.front();
        for (int32_t h : ts[i].cand)
            if (load[h] < load[best]) best = h;
        host[i] = best;
        load[best] += ts[i].dur;
    }
    return list_schedule(ts, order, host, nhosts);
}

// Lower bound (Eq. 4 style): no host finishes before the work it must do.
int64_t lower_bound(const std::vector<STask> &ts, int nhosts) {
    std::vector<int64_t> must(nhosts, 0);
    int64_t lb = 0;
    for (const auto &t : ts) {
        for (int32_t r : t.recv) must[r] += t.dur;
        if (t.cand.size() == 1) must[t.cand[0]] += t.dur;
        lb = std::max(lb, t.dur);
    }
    for (int64_t m : must) lb = std::max(lb, m);
    return lb;
}

// Depth-first search over (next task, its sender host) with pruning by a
// per-host lower bound; tasks identical in duration, candidates and
// receivers are interchangeable, so only the first unscheduled one of each
// class is branched on.  Stops after max_nodes branches; returns the best
// schedule seen, starting from the load-balance schedule.
struct Dfs {
    const std::vector<STask> &ts;
    int nhosts;
    int64_t max_nodes;
    int64_t nodes = 0;
    std::vector<int32_t> cls;  // class id per task
    std::vector<char> done;
    std::vector<int32_t> order, host;
    std::vector<int64_t> free_at, must;  // must: remaining certain work per host
    Sched best;

    void run(std::vector<int32_t> &cur_order, std::vector<int32_t> &cur_host, int64_t span) {
        const size_t n = ts.size();
        if (cur_order.size() == n) {
            if (span < best.makespan) {
                best = list_schedule(ts, cur_order, cur_host, nhosts);
            }
            return;
        }
        std::vector<char> seen_cls(n, 0);
        for (size_t i = 0; i < n; ++i) {
            if (done[i] || seen_cls[cls[i]]) continue;
            seen_cls[cls[i]] = 1;
            const STask &t = ts[i];
            for (int32_t h : t.cand) {
                if (nodes >= max_nodes) return;
                ++nodes;
                int64_t st = free_at[h];
                for (int32_t r : t.recv) st = std::max(st, free_at[r]);
                const int64_t fin = st + t.dur;
                // apply
                const int64_t old_h = free_at[h];
                std::vector<int64_t> old_r(t.recv.size());
                for (size_t k = 0; k < t.recv.size(); ++k) old_r[k] = free_at[t.recv[k]];
                free_at[h] = fin;
                for (int32_t r : t.recv) free_at[r] = fin;
                for (int32_t r : t.recv) must[r] -= t.dur;
                if (t.cand.size() == 1) must[h] -= t.dur;
                int64_t lb = std::max(span, fin);
                for (int q = 0; q < nhosts; ++q) lb = std::max(lb, free_at[q] + must[q]);
                if (lb < best.makespan) {
                    done[i] = 1;
                    cur_order.push_back(int32_t(i));
                    cur_host[i] = h;
                    run(cur_order, cur_host, std::max(span, fin));
                    cur_order.pop_back();
                    done[i] = 0;
                }
                // undo
                if (t.cand.size() == 1) must[h] += t.dur;
                for (int32_t r : t.recv) must[r] += t.dur;
                for (size_t k = 0; k < t.recv.size(); ++k) free_at[t.recv[k]] = old_r[k];
                free_at[h] = old_h;
            }
        }
    }
};

Sched dfs(const std::vector<STask> &ts, int nhosts, int64_t max_nodes, int64_t *nodes_out) {
    Dfs d{ts, nhosts, max_nodes, 0, {}, {}, {}, {}, {}, {}, {}};
    const size_t n = ts.size();
    d.cls.assign(n, 0);
    for (size_t i = 0; i < n; ++i) {
        d.cls[i] = int32_t(i);
        for (size_t j = 0; j < i; ++j)
            if (ts[j].dur == ts[i].dur && ts[j].cand == ts[i].cand && ts[j].recv == ts[i].recv) {
                d.cls[i] = d.cls[j];
                break;
            }
    }
    d.done.assign(n, 0);
    d.free_at.assign(nhosts, 0);
    d.must.assign(nhosts, 0);
    for (const auto &t : ts) {
        for (int32_t r : t.recv) d.must[r] += t.dur;
        if (t.cand.size() == 1) d.must[t.cand[0]] += t.dur;
    }
    d.best = load_balance(ts, nhosts);
    std::vector<int32_t> cur_order, cur_host(n, -1);
    d.run(cur_order, cur_host, 0);
    if (nodes_out) *nodes_out = d.nodes;
    return d.best;
}

// Greedy search with randomization: from the current time, repeatedly draw
// random orders of the unscheduled tasks, take each task whose receivers and
// some candidate sender host (lowest free one) are idle, keep the set that
// keeps the most hosts busy (first best), start it, and advance to the next
// finish.
Sched randomized(const std::vector<STask> &ts, int nhosts, int64_t rounds, uint64_t seed) {
    const size_t n = ts.size();
    Sched s;
    s.host.assign(n, -1);
    s.start.assign(n, 0);
    SplitMix64 rng{seed};
    std::vector<int32_t> remaining(n);
    for (size_t i = 0; i < n; ++i) remaining[i] = int32_t(i);
    std::vector<int64_t> busy_until(nhosts, 0);
    int64_t now = 0;
    while (!remaining.empty()) {
        std::vector<int32_t> best_set, best_host;
        int best_score = -1;
        for (int64_t r = 0; r < std::max<int64_t>(1, rounds); ++r) {
            std::vector<int32_t> perm = remaining;
            for (size_t i = perm.size(); i > 1; --i) {
                const size_t j = size_t(rng.next() % uint64_t(i));
                std::swap(perm[i - 1], perm[j]);
            }
            std::vector<char> used(nhosts, 0);
            for (int q = 0; q < nhosts; ++q) used[q] = busy_until[q] > now;
            std::vector<int32_t> set, hosts;
            int score = 0;
            for (int32_t i : perm) {
                bool ok = true;
                for (int32_t rh : ts[i].recv) ok = ok && !used[rh];
                if (!ok) continue;
                int32_t h = -1;
                for (int32_t c : ts[i].cand)
                    if (!used[c]) { h = c; break; }
                if (h < 0) continue;
                used[h] = 1;
                for (int32_t rh : ts[i].recv) used[rh] = 1;
                set.push_back(i);
                hosts.push_back(h);
                score += 1 + int(ts[i].recv.size());
            }
            if (score > best_score) {
                best_score = score;
                best_set = set;
                best_host = hosts;
            }
        }
        for (size_t k = 0; k < best_set.size(); ++k) {
            const int32_t i = best_set[k], h = best_host[k];
            s.host[i] = h;
            s.start[i] = now;
            const int64_t fin = now + ts[i].dur;
            busy_until[h] = fin;
            for (int32_t rh : ts[i].recv) busy_until[rh] = fin;
            s.makespan = std::max(s.makespan, fin);
        }
        std::vector<int32_t> rest;
        for (int32_t i : remaining)
            if (std::find(best_set.begin(), best_set.end(), i) == best_set.end()) rest.push_back(i);
        remaining.swap(rest);
        if (remaining.empty()) break;
        int64_t next = INT64_MAX;  // next finish after now
        for (int q = 0; q < nhosts; ++q)
            if (busy_until[q] > now) next = std::min(next, busy_until[q]);
        if (next != INT64_MAX) now = next;
    }
    return s;
}

}  // namespace
}  // namespace rs

extern "C" reshard_status_t reshard_schedule(const reshard_plan_t *plan, int64_t src_devices_per_host,
                                             int64_t dst_devices_per_host, reshard_sched_algo_t algo,
                                             int64_t max_dfs_nodes, int64_t random_rounds, uint64_t seed,
                                             int64_t *sender_out, int64_t *start_out, int64_t *makespan_out,
                                             int64_t *lower_bound_out, int64_t *dfs_nodes_out) {
    return rs::guarded([&]() -> reshard_status_t {
        using namespace rs;
        const Plan *p = reinterpret_cast<const Plan *>(plan);
        if (!p) return fail(RESHARD_EINVAL, "NULL plan");
        if (src_devices_per_host < 1 || dst_devices_per_host < 1)
            return fail(RESHARD_EINVAL, "devices per host must be >= 1");
        if (max_dfs_nodes < 0 || random_rounds < 0) return fail(RESHARD_EINVAL, "negative budget");
        if (int(algo) < 0 || int(algo) > 4) return fail(RESHARD_EINVAL, "unknown scheduling algorithm");
        const int hs = int((p->src.ndev + src_devices_per_host - 1) / src_devices_per_host);
        const int hd = int((p->dst.ndev + dst_devices_per_host - 1) / dst_devices_per_host);
        const int nhosts = hs + hd;
        std::vector<STask> ts(p->tasks.size());
        for (size_t i = 0; i < p->tasks.size(); ++i) {
            const UnitTask &t = p->tasks[i];
            ts[i].dur = t.bytes;
            std::set<int32_t> c, r;
            for (int64_t k = p->src.shard_devs_off[t.src_shard]; k < p->src.shard_devs_off[t.src_shard + 1]; ++k)
                c.insert(int32_t(p->src.shard_devs[k] / src_devices_per_host));
            for (int64_t k = p->dst.shard_devs_off[t.dst_shard]; k < p->dst.shard_devs_off[t.dst_shard + 1]; ++k)
                r.insert(int32_t(hs + p->dst.shard_devs[k] / dst_devices_per_host));
            ts[i].cand.assign(c.begin(), c.end());
            ts[i].recv.assign(r.begin(), r.end());
        }
        Sched s;
        int64_t nodes = 0;
        switch (algo) {
            case RESHARD_SCHED_NAIVE: s = naive(ts, nhosts); break;
            case RESHARD_SCHED_LOAD_BALANCE: s = load_balance(ts, nhosts); break;
            case RESHARD_SCHED_DFS: s = dfs(ts, nhosts, max_dfs_nodes, &nodes); break;
            case RESHARD_SCHED_RANDOMIZED: s = randomized(ts, nhosts, random_rounds, seed); break;
            case RESHARD_SCHED_ENSEMBLE: {
                const Sched a = dfs(ts, nhosts, max_dfs_nodes, &nodes);
                const Sched b = randomized(ts, nhosts, random_rounds, seed);
                s = b.makespan < a.makespan ? b : a;
                break;
            }
        }
        for (size_t i = 0; i < p->tasks.size(); ++i) {
            // the sender device: the task's lowest-indexed owner on the chosen host
            const UnitTask &t = p->tasks[i];
            int64_t dev = -1;
            for (int64_t k = p->src.shard_devs_off[t.src_shard]; k < p->src.shard_devs_off[t.src_shard + 1]; ++k)
                if (p->src.shard_devs[k] / src_devices_per_host == s.host[i]) {
                    dev = p->src.shard_devs[k];
                    break;
                }
            if (sender_out) sender_out[i] = dev;
            if (start_out) start_out[i] = s.start[i];
        }
        if (makespan_out) *makespan_out = s.makespan;
        if (lower_bound_out) *lower_bound_out = lower_bound(ts, nhosts);
        if (dfs_nodes_out) *dfs_nodes_out = nodes;
        return RESHARD_OK;
    });
}
