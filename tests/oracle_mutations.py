"""Plausible mistakes planted in the oracle, on the CPU, to show that its pins
catch them (tests/test_oracle_mutations.py).  `apply(name)` replaces one
oracle function, in the module and in the package namespace, for the rest
of the process; tests/conftest.py calls it when RESHARD_ORACLE_MUTATION
names a mutation.  Nothing here is used by a normal test run."""

import importlib
import itertools

import numpy as np

import oracle

# the module itself: the package re-exports the function `reshard` under the
# submodule's name, so `import oracle.reshard as R` would bind that function
R = importlib.import_module("oracle.reshard")
SCH = importlib.import_module("oracle.schedule")
PIPE = importlib.import_module("oracle.pipeline")
SCH._DFS = SCH.dfs  # the unmutated search, for the first-descent mutation


def _split_ceil(length, k):
    # padding-style split: ceil-sized shards first, the last one short
    c = -(-length // k) if k else 0
    return [(min(j * c, length), min((j + 1) * c, length)) for j in range(k)]


def _split_remainder_last(length, k):
    # the longer shards at the end instead of the start
    q, r = divmod(length, k)
    out, lo = [], 0
    for j in range(k):
        n = q + (1 if j >= k - r else 0)
        out.append((lo, lo + n))
        lo += n
    return out


def _shard_index_minor_major(coords, axes, mesh):
    j = 0
    for a in reversed(tuple(axes)):
        j = j * mesh[a] + coords[a]
    return j


def _device_coords_column_major(mesh, device):
    return tuple(int(c) for c in np.unravel_index(device, tuple(mesh), order="F"))


def _lpt_shortest_first(tasks, itemsize, n_src_devices):
    load = [0] * n_src_devices
    chosen = [None] * len(tasks)
    for i in sorted(range(len(tasks)), key=lambda i: (R._task_bytes(tasks[i], itemsize), i)):
        pick = min(tasks[i]["senders"], key=lambda k: (load[k], k))
        chosen[i] = pick
        load[pick] += R._task_bytes(tasks[i], itemsize)
    return chosen


def _lpt_heaviest_sender(tasks, itemsize, n_src_devices):
    load = [0] * n_src_devices
    chosen = [None] * len(tasks)
    for i in sorted(range(len(tasks)), key=lambda i: (-R._task_bytes(tasks[i], itemsize), i)):
        pick = max(tasks[i]["senders"], key=lambda k: (load[k], -k))
        chosen[i] = pick
        load[pick] += R._task_bytes(tasks[i], itemsize)
    return chosen


def _naive_highest(tasks):
    return [max(t["senders"]) for t in tasks]


def _unit_tasks_source_cuts_only(shape, src_mesh, src_spec, dst_mesh, dst_spec):
    # the destination layout's shard boundaries left out of the cut points
    shape = tuple(shape)
    sdims = R.parse_spec(src_spec, len(shape), len(src_mesh))
    ddims = R.parse_spec(dst_spec, len(shape), len(dst_mesh))
    intervals = []
    for d, length in enumerate(shape):
        cuts = {0, length}
        for lo, hi in R.split_bounds(length, R.shard_count(sdims[d], src_mesh)):
            cuts.update((lo, hi))
        pts = sorted(cuts)
        intervals.append([(a, b) for a, b in zip(pts[:-1], pts[1:]) if b > a])
    sboxes = [R.device_box(shape, src_mesh, sdims, k) for k in range(R._n_devices(src_mesh))]
    dboxes = [R.device_box(shape, dst_mesh, ddims, k) for k in range(R._n_devices(dst_mesh))]

    def owns(box, sl):
        return all(blo <= lo and hi <= bhi for (blo, bhi), (lo, hi) in zip(box, sl))

    return [{"box": tuple(sl), "senders": [k for k, b in enumerate(sboxes) if owns(b, sl)],
             "receivers": [k for k, b in enumerate(dboxes) if owns(b, sl)]}
            for sl in itertools.product(*intervals)]


def _unshard_without_replica_check(shards, shape, mesh, spec):
    shape = tuple(shape)
    dims = R.parse_spec(spec, len(shape), len(mesh))
    itemsize = np.asarray(shards[0]).dtype.itemsize
    x = np.zeros(shape, dtype=np.dtype(f"u{itemsize}"))
    for d, s in enumerate(shards):
        x[R._slices(R.device_box(shape, mesh, dims, d))] = R._bits(np.asarray(s))
    return x


def _traffic_unique_writes(shape, itemsize, dst_mesh, dst_spec):
    # replicas counted once
    n = int(np.prod(shape, dtype=np.int64)) if len(shape) else 1
    return n * itemsize, n * itemsize


_PARSE = R.parse_spec


def _parse_spec_first_axis_only(spec, ndim, mesh_ndim):
    # a multi-axis token such as S^{01} keeps only its first axis
    return tuple(tuple(axes[:1]) for axes in _PARSE(spec, ndim, mesh_ndim))


def _parse_spec_axes_reversed(spec, ndim, mesh_ndim):
    # S^{01} read as S^{10}
    return tuple(tuple(reversed(axes)) for axes in _PARSE(spec, ndim, mesh_ndim))


_SHARD = R.shard


def _shard_inverse_perm(x, mesh, spec, perm=None):
    # the buffer laid out with the inverse permutation
    if perm is not None:
        perm = tuple(int(a) for a in np.argsort(perm))
    return _SHARD(x, mesh, spec, perm)


def _shard_perm_reshape(x, mesh, spec, perm=None):
    # the buffer reshaped to the permuted extents instead of transposed
    plain = _SHARD(x, mesh, spec)
    if perm is None:
        return plain
    perm = R.check_perm(perm, x.ndim)
    return [np.ascontiguousarray(a.reshape(tuple(a.shape[k] for k in perm))) for a in plain]


_UNSHARD = R.unshard


def _unshard_perm_reshape(shards, shape, mesh, spec, perm=None):
    # permuted buffers reshaped back to the box instead of transposed
    if perm is None:
        return _UNSHARD(shards, shape, mesh, spec)
    dims = R.parse_spec(spec, len(shape), len(mesh))
    plain = []
    for d, s in enumerate(shards):
        box = R.device_box(tuple(shape), mesh, dims, d)
        plain.append(np.asarray(s).reshape(tuple(hi - lo for lo, hi in box)))
    return _UNSHARD(plain, shape, mesh, spec)


_LOCAL_SHAPE = R.local_shape


def _local_shape_unpermuted(shape, mesh, spec, device, perm=None):
    # the box's extents in tensor order whatever the buffer's order
    return _LOCAL_SHAPE(shape, mesh, spec, device)


# scheduling across hosts (Section 3.2)

def _start_times_sender_only(model, order, host):
    # a task waits for earlier tasks on its sender host only, not for its receivers
    start = [None] * len(model)
    for pos, i in enumerate(order):
        s = 0
        for j in order[:pos]:
            if host[j] == host[i]:
                s = max(s, start[j] + model[j][0])
        start[i] = s
    return start


def _start_times_serial(model, order, host):
    # every task waits for every earlier task
    start, t = [None] * len(model), 0
    for i in order:
        start[i] = t
        t += model[i][0]
    return start


def _lower_bound_all_candidates(model, nhosts):
    # every candidate sender charged as if it had to send
    must = [0] * nhosts
    lb = 0
    for dur, cand, recv in model:
        for h in list(recv) + list(cand):
            must[h] += dur
        lb = max(lb, dur)
    return max([lb] + must)


def _load_balance_shortest_first(model, nhosts):
    order = sorted(range(len(model)), key=lambda i: (model[i][0], i))
    load = [0] * nhosts
    host = [None] * len(model)
    for i in order:
        best = min(model[i][1], key=lambda h: (load[h], h))
        host[i] = best
        load[best] += model[i][0]
    return SCH.schedule(model, order, host)


def _randomized_without_search(model, nhosts, rounds, seed):
    # no random orders at all: the load-balance schedule
    return SCH.load_balance(model, nhosts)


_RANDOMIZED = SCH.randomized


def _randomized_one_round(model, nhosts, rounds, seed):
    # a single random order per iteration: no search for the largest set
    return _RANDOMIZED(model, nhosts, 1, seed)


def _dfs_first_descent(model, nhosts, max_nodes):
    # the search stops at its first complete schedule
    return SCH.__dict__["_DFS"](model, nhosts, 1)


# pipeline schedules (Section 4)

def _stage_ops_warmup_plus_one(S, M, s, eager):
    i = s + 1
    w = 2 * (S - i) + 1 if eager else S - i + 2
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


_STAGE_OPS = PIPE.stage_ops


def _stage_ops_eager_ignored(S, M, s, eager):
    return _STAGE_OPS(S, M, s, False)


# name: (module, function, replacement, pin file, -k selection of its pins)
_PINS_R = ("test_oracle_pins.py", None)
_PINS_S = ("test_schedule.py", "not library and not errors and not golden")
_PINS_P = ("test_pipeline.py", "not parity and not errors")
MUTATIONS = {
    "split_ceil": (R, "split_bounds", _split_ceil, _PINS_R),
    "split_remainder_last": (R, "split_bounds", _split_remainder_last, _PINS_R),
    "shard_index_minor_major": (R, "shard_index", _shard_index_minor_major, _PINS_R),
    "device_coords_column_major": (R, "device_coords", _device_coords_column_major, _PINS_R),
    "lpt_shortest_first": (R, "choose_senders_lpt", _lpt_shortest_first, _PINS_R),
    "lpt_heaviest_sender": (R, "choose_senders_lpt", _lpt_heaviest_sender, _PINS_R),
    "naive_highest": (R, "choose_senders_naive", _naive_highest, _PINS_R),
    "unit_tasks_source_cuts_only": (R, "unit_tasks", _unit_tasks_source_cuts_only, _PINS_R),
    "unshard_without_replica_check": (R, "unshard", _unshard_without_replica_check, _PINS_R),
    "traffic_unique_writes": (R, "traffic_bytes", _traffic_unique_writes, _PINS_R),
    "shard_inverse_perm": (R, "shard", _shard_inverse_perm, _PINS_R),
    "shard_perm_reshape": (R, "shard", _shard_perm_reshape, _PINS_R),
    "unshard_perm_reshape": (R, "unshard", _unshard_perm_reshape, _PINS_R),
    "local_shape_unpermuted": (R, "local_shape", _local_shape_unpermuted, _PINS_R),
    "parse_spec_first_axis_only": (R, "parse_spec", _parse_spec_first_axis_only, _PINS_R),
    "parse_spec_axes_reversed": (R, "parse_spec", _parse_spec_axes_reversed, _PINS_R),
    "start_times_sender_only": (SCH, "start_times", _start_times_sender_only, _PINS_S),
    "start_times_serial": (SCH, "start_times", _start_times_serial, _PINS_S),
    "lower_bound_all_candidates": (SCH, "lower_bound", _lower_bound_all_candidates, _PINS_S),
    "load_balance_shortest_first": (SCH, "load_balance", _load_balance_shortest_first, _PINS_S),
    "randomized_without_search": (SCH, "randomized", _randomized_without_search, _PINS_S),
    "randomized_one_round": (SCH, "randomized", _randomized_one_round, _PINS_S),
    "dfs_first_descent": (SCH, "dfs", _dfs_first_descent, _PINS_S),
    "pipeline_warmup_plus_one": (PIPE, "stage_ops", _stage_ops_warmup_plus_one, _PINS_P),
    "pipeline_eager_ignored": (PIPE, "stage_ops", _stage_ops_eager_ignored, _PINS_P),
}


def apply(name):
    module, fn_name, fn, _ = MUTATIONS[name]
    setattr(module, fn_name, fn)
    if module is R and hasattr(oracle, fn_name):
        setattr(oracle, fn_name, fn)
