"""Element-by-element brute force for tiny reshards (test helper).

A second formulation of the layout semantics, used to pin the oracle.  It
never builds boxes: for every logical index it asks, dimension by dimension,
which shard numpy.array_split puts that index into, turns the shard number
back into the mesh coordinates that must hold it (mixed-radix digits, most
significant axis first) and places the element at its rank inside that
shard.  Pure Python on small inputs only.
"""

import itertools

import numpy as np


def _digits(j, radices):
    """Mixed-radix digits of j, most significant first."""
    out = []
    for r in reversed(radices):
        out.append(j % r)
        j //= r
    return tuple(reversed(out))


def _owner_tables(length, k):
    """For each index: (shard number, rank inside the shard), via numpy.array_split."""
    owner = [None] * length
    for j, piece in enumerate(np.array_split(np.arange(length), k)):
        for rank, i in enumerate(piece.tolist()):
            owner[i] = (j, rank)
    return owner


def layout(x, mesh, dims, perm=None):
    """Per-device arrays of ``x`` under (mesh, per-dim axis tuples), element by
    element; with ``perm``, buffer index k is the element's rank along tensor
    dimension perm[k]."""
    perm = tuple(range(x.ndim)) if perm is None else tuple(perm)
    shape = x.shape
    ndev = int(np.prod(mesh))
    coords = [tuple(int(c) for c in np.unravel_index(d, mesh)) for d in range(ndev)]
    tables = []
    for length, axes in zip(shape, dims):
        k = int(np.prod([mesh[a] for a in axes])) if axes else 1
        tables.append(_owner_tables(length, k))

    def holds(dev, d, i):
        j, _ = tables[d][i]
        axes = dims[d]
        if not axes:
            return True
        want = _digits(j, [mesh[a] for a in axes])
        return all(coords[dev][a] == w for a, w in zip(axes, want))

    out = []
    for dev in range(ndev):
        per_dim = [[i for i in range(shape[d]) if holds(dev, d, i)] for d in range(len(shape))]
        local = np.zeros(tuple(len(per_dim[a]) for a in perm), dtype=x.dtype)
        for idx in itertools.product(*per_dim):
            rank = [tables[d][i][1] for d, i in enumerate(idx)]
            local[tuple(rank[a] for a in perm)] = x[idx]
        out.append(local)
    return out
