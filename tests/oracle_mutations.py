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


MUTATIONS = {
    "split_ceil": ("split_bounds", _split_ceil),
    "split_remainder_last": ("split_bounds", _split_remainder_last),
    "shard_index_minor_major": ("shard_index", _shard_index_minor_major),
    "device_coords_column_major": ("device_coords", _device_coords_column_major),
    "lpt_shortest_first": ("choose_senders_lpt", _lpt_shortest_first),
    "lpt_heaviest_sender": ("choose_senders_lpt", _lpt_heaviest_sender),
    "naive_highest": ("choose_senders_naive", _naive_highest),
    "unit_tasks_source_cuts_only": ("unit_tasks", _unit_tasks_source_cuts_only),
    "unshard_without_replica_check": ("unshard", _unshard_without_replica_check),
    "traffic_unique_writes": ("traffic_bytes", _traffic_unique_writes),
}


def apply(name):
    fn_name, fn = MUTATIONS[name]
    setattr(R, fn_name, fn)
    if hasattr(oracle, fn_name):
        setattr(oracle, fn_name, fn)
