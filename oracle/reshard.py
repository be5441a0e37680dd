"""Oracle for one cross-mesh resharding task (numpy, CPU) -- test infrastructure.

Nothing here is used by the product path: only ``tests/``,
``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg import it.

What is computed (paper, Section 2.2, "Cross-mesh resharding"): a tensor D
laid out on a source mesh under spec X_A is re-laid out on a disjoint
destination mesh under spec X_B.  The result is fully determined by the two
layouts, so the oracle is the plain definition: rebuild the logical tensor
from the source shards, then cut it again under the destination layout.
Every copy works on raw-bit views (unsigned integers of the element size),
so NaN payloads, signed zeros and infinities pass through untouched.

Readings of the paper used below (the paper is silent or garbled there):

* Device numbering is row-major over mesh coordinates (Section 2.2, "Device
  mesh": the (2,2) mesh is [[0,1],[2,3]]).
* A sharded dimension "S^{a1 a2 ..}" splits over the listed mesh axes in
  the listed order, the first axis being the most significant digit of the
  shard index ("axis-list-major"; for S^{01} the shard is c0*m1 + c1).
  Mesh axes used by no dimension replicate (Section 2.2, "Sharding spec").
  A mesh axis may appear at most once in a spec.
* A length l cut into k shards uses the balanced split: shard j starts at
  j*floor(l/k) + min(j, l mod k), so the first (l mod k) shards are one
  element longer (66 into 4 gives 17,17,16,16).  For even lengths this is
  the appendix's "k equal size" cut at l/k, 2l/k, ...  No padding is stored.
* Each device's local buffer is the dense C-order array of its box.  The
  paper's specs never permute dimensions; a local layout may optionally be
  permuted (an extension for transposed layouts, not in the paper): with
  perm = (p_0, ..., p_{n-1}), dimension k of the buffer is tensor dimension
  p_k, i.e. the buffer is numpy.transpose(box, perm).  None is the identity.

Parity pins (see tests/test_oracle_pins.py): brute-force per-element
ownership on tiny meshes, the Fig. 2 facts stated in Section 2.2, the
Table 3 unit-task counts stated in Section 5.1.2 and Section 5.3.1,
numpy.array_split, and the invariants reassembly / replica identity /
identity-copy / round trip / traffic lower bound (Section 2.2) /
composition.  The LPT sender choice is pinned by brute force over all
assignments of Eq. 4 on small task sets.
"""

from __future__ import annotations

import itertools
import re

import numpy as np

# ---------------------------------------------------------------------------
# Layout definitions (Section 2.2)
# ---------------------------------------------------------------------------

_TOKEN = re.compile(r"R|S[\^_]?(\{[0-9]+\}|[0-9]+)")


def parse_spec(spec, ndim, mesh_ndim):
    """Sharding spec string -> tuple (per tensor dim) of mesh-axis tuples.

    Section 2.2, "Sharding spec": an N-letter string X_0^{d_0} ... with
    X_i in {S, R}; S carries the mesh dimensions the tensor dimension is
    sharded along.  R gives the empty tuple.  Accepted spellings include
    ``S^0RR``, ``RS^{01}R``, ``S_{0}RR`` and ``S0 R S1``; spaces and commas
    between letters are ignored.
    """
    text = spec.replace(" ", "").replace(",", "")
    pos = 0
    dims = []
    while pos < len(text):
        m = _TOKEN.match(text, pos)
        if m is None:
            raise ValueError(f"bad sharding spec {spec!r} at {text[pos:]!r}")
        tok = m.group(0)
        if tok == "R":
            dims.append(())
        else:
            digits = m.group(1).strip("{}")
            dims.append(tuple(int(c) for c in digits))
        pos = m.end()
    if len(dims) != ndim:
        raise ValueError(f"spec {spec!r} has {len(dims)} letters, tensor has {ndim} dims")
    used = [a for axes in dims for a in axes]
    for a in used:
        if a >= mesh_ndim:
            raise ValueError(f"spec {spec!r} names mesh axis {a}, mesh has {mesh_ndim} axes")
    if len(set(used)) != len(used):
        raise ValueError(f"spec {spec!r} uses a mesh axis twice")
    return tuple(dims)


def split_bounds(length, k):
    """[lo, hi) of each of the k shards of a dimension of the given length.

    Balanced split (reading of the appendix's "k equal size" cut and of the
    padding remark in Section 5.1): shard j starts at j*(l//k) + min(j, l%k).
    """
    q, r = divmod(length, k)
    out = []
    for j in range(k):
        lo = j * q + min(j, r)
        hi = lo + q + (1 if j < r else 0)
        out.append((lo, hi))
    return out


def device_coords(mesh, device):
    """Row-major mesh coordinates of a device index (Section 2.2, "Device mesh")."""
    return tuple(int(c) for c in np.unravel_index(device, tuple(mesh)))


def shard_index(coords, axes, mesh):
    """Shard number along one tensor dim for a device at ``coords``.

    The axes are read major to minor: for axes (a1, a2) the index is
    c[a1]*m[a2] + c[a2].  The total shard count is the product of m[a].
    """
    j = 0
    for a in axes:
        j = j * mesh[a] + coords[a]
    return j


def shard_count(axes, mesh):
    k = 1
    for a in axes:
        k *= mesh[a]
    return k


def device_box(shape, mesh, dims, device):
    """Per-dimension [lo, hi) of the data slice held by ``device`` (Section 2.2, "Data slice")."""
    coords = device_coords(mesh, device)
    box = []
    for length, axes in zip(shape, dims):
        k = shard_count(axes, mesh)
        box.append(split_bounds(length, k)[shard_index(coords, axes, mesh)])
    return tuple(box)


def check_perm(perm, ndim):
    """The identity for None; else perm must order 0..ndim-1."""
    if perm is None:
        return tuple(range(ndim))
    perm = tuple(int(a) for a in perm)
    if sorted(perm) != list(range(ndim)):
        raise ValueError(f"{perm} is not a permutation of the {ndim} tensor dimensions")
    return perm


def local_shape(shape, mesh, spec, device, perm=None):
    """Shape of ``device``'s buffer: its box's extents, in the order of ``perm``."""
    dims = parse_spec(spec, len(shape), len(mesh))
    ext = tuple(hi - lo for lo, hi in device_box(shape, mesh, dims, device))
    return tuple(ext[a] for a in check_perm(perm, len(shape)))


def _n_devices(mesh):
    n = 1
    for m in mesh:
        n *= m
    return n


def _bits(a):
    """Raw-bit view of an array: unsigned integers of the same item size."""
    a = np.ascontiguousarray(a)
    return a.view({1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}[a.dtype.itemsize])


def _slices(box):
    return tuple(slice(lo, hi) for lo, hi in box)


# ---------------------------------------------------------------------------
# The result of a resharding task (Section 2.2)
# ---------------------------------------------------------------------------

def shard(x, mesh, spec, perm=None):
    """Lay the logical tensor ``x`` out on ``mesh`` under ``spec``.

    Returns one dense C-order array per device, in row-major device order:
    the device's box, its dimensions ordered by ``perm``.  Replicated
    devices get equal, separate copies.
    """
    dims = parse_spec(spec, x.ndim, len(mesh))
    perm = check_perm(perm, x.ndim)
    return [np.ascontiguousarray(np.transpose(x[_slices(device_box(x.shape, mesh, dims, d))], perm)).copy()
            for d in range(_n_devices(mesh))]


def unshard(shards, shape, mesh, spec, perm=None):
    """Rebuild the logical tensor from per-device shards (buffers laid out
    in the order of ``perm``).

    Every element must be covered; where replicas overlap their bits must
    agree (otherwise the input is not a valid layout and ValueError is
    raised).  Works on raw-bit views and returns a raw-bit array.
    """
    shape = tuple(shape)
    dims = parse_spec(spec, len(shape), len(mesh))
    perm = check_perm(perm, len(shape))
    back = tuple(int(a) for a in np.argsort(perm))  # buffer dimension holding tensor dimension d
    if len(shards) != _n_devices(mesh):
        raise ValueError("need one shard per mesh device")
    itemsize = np.asarray(shards[0]).dtype.itemsize
    x = np.zeros(shape, dtype=np.dtype(f"u{itemsize}"))
    filled = np.zeros(shape, dtype=bool)
    for d, s in enumerate(shards):
        box = device_box(shape, mesh, dims, d)
        want = tuple(hi - lo for lo, hi in box)
        s = _bits(np.asarray(s))
        if s.shape != tuple(want[a] for a in perm):
            raise ValueError(f"device {d}: shard shape {s.shape}, layout needs {tuple(want[a] for a in perm)}")
        s = np.transpose(s, back)
        sl = _slices(box)
        seen = filled[sl]
        if seen.any() and not np.array_equal(x[sl][seen], s[seen]):
            raise ValueError(f"device {d}: replica disagrees with an earlier copy")
        x[sl] = s
        filled[sl] = True
    if not filled.all():
        raise ValueError("source layout does not cover the tensor")
    return x


def reshard(src_shards, shape, src_mesh, src_spec, dst_mesh, dst_spec, src_perm=None, dst_perm=None):
    """Destination shards of one cross-mesh resharding task.

    Section 2.2: D, laid out on the source mesh under src_spec, is sent to
    the destination mesh where its layout becomes dst_spec.  Computed as
    unshard-then-shard on raw bits; the output arrays carry the dtype of the
    inputs (bit-identical).  The optional permutations order each side's
    buffer dimensions (see the module header).
    """
    dtype = np.asarray(src_shards[0]).dtype
    x = unshard(src_shards, shape, src_mesh, src_spec, src_perm)
    return [s.view(dtype) for s in shard(x, dst_mesh, dst_spec, dst_perm)]


def traffic_bytes(shape, itemsize, dst_mesh, dst_spec):
    """Algorithmic bytes of one reshard: (read, written).

    Read: the tensor once -- the lower bound on the message size stated in
    Section 2.2.  Written: every destination device's local shard, so
    replicated destinations count once per replica.
    """
    n = int(np.prod(shape, dtype=np.int64)) if len(shape) else 1
    written = 0
    for d in range(_n_devices(dst_mesh)):
        written += int(np.prod(local_shape(shape, dst_mesh, dst_spec, d), dtype=np.int64))
    return n * itemsize, written * itemsize


# ---------------------------------------------------------------------------
# Unit communication tasks (Section 2.2 and appendix "Algorithm to decompose")
# ---------------------------------------------------------------------------

def unit_tasks(shape, src_mesh, src_spec, dst_mesh, dst_spec):
    """Unit tasks of a resharding, following the appendix decomposition.

    For every tensor dimension the cut points are {0, l} plus the shard
    boundaries of the source layout and of the destination layout; the
    intervals between consecutive distinct cut points form the per-dim
    interval sets, and their cross product is the slice set.  Each slice's
    senders are all source devices owning it and its receivers are all
    destination devices requiring it.  Slices come out in lexicographic
    order of their lower corner.

    Returns a list of dicts: {"box": ((lo,hi),...), "senders": [...],
    "receivers": [...]}.
    """
    shape = tuple(shape)
    sdims = parse_spec(src_spec, len(shape), len(src_mesh))
    ddims = parse_spec(dst_spec, len(shape), len(dst_mesh))
    intervals = []
    for d, length in enumerate(shape):
        cuts = {0, length}
        for dims, mesh in ((sdims, src_mesh), (ddims, dst_mesh)):
            for lo, hi in split_bounds(length, shard_count(dims[d], mesh)):
                cuts.add(lo)
                cuts.add(hi)
        pts = sorted(cuts)
        intervals.append([(a, b) for a, b in zip(pts[:-1], pts[1:]) if b > a])
    sboxes = [device_box(shape, src_mesh, sdims, k) for k in range(_n_devices(src_mesh))]
    dboxes = [device_box(shape, dst_mesh, ddims, k) for k in range(_n_devices(dst_mesh))]

    def owns(box, sl):
        return all(blo <= lo and hi <= bhi for (blo, bhi), (lo, hi) in zip(box, sl))

    tasks = []
    for sl in itertools.product(*intervals):
        tasks.append({
            "box": tuple(sl),
            "senders": [k for k, b in enumerate(sboxes) if owns(b, sl)],
            "receivers": [k for k, b in enumerate(dboxes) if owns(b, sl)],
        })
    return tasks


def _task_bytes(task, itemsize):
    v = 1
    for lo, hi in task["box"]:
        v *= hi - lo
    return v * itemsize


def choose_senders_naive(tasks):
    """Section 3.2, "Naive algorithm": the lowest-indexed owner sends."""
    return [min(t["senders"]) for t in tasks]


def choose_senders_lpt(tasks, itemsize, n_src_devices):
    """Section 3.2, "Load balance only" (Eq. 4): greedy longest-first.

    Tasks are visited in descending order of duration T_i (taken as the
    slice's byte count; ties keep the task order), and each goes to the
    candidate sender with the lightest load so far (ties: lowest device
    index).  Balancing is per device: one GPU has no hosts to group by.
    """
    load = [0] * n_src_devices
    chosen = [None] * len(tasks)
    order = sorted(range(len(tasks)), key=lambda i: (-_task_bytes(tasks[i], itemsize), i))
    for i in order:
        pick = min(tasks[i]["senders"], key=lambda k: (load[k], k))
        chosen[i] = pick
        load[pick] += _task_bytes(tasks[i], itemsize)
    return chosen
