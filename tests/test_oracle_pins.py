"""Pins of the CPU oracle against facts that do not come from the oracle itself.

* numpy.array_split (library) and the 17,17,16,16 split of H=66 named for the
  U-Transformer skip-tensor workload;
* the facts Section 2.2 states about Fig. 2 (tests/golden/fig2_device_view.json);
* the unit-task counts the paper states for Table 3 cases 4 and 8
  (tests/golden/table3_cases.json);
* an element-by-element brute force (tests/bruteforce.py) on tiny meshes;
* invariants: reassembly, replica identity, identity reshard is a copy,
  round trip, traffic lower bound (Section 2.2), composition A->B->C == A->C;
* the LPT sender choice (Section 3.2, Eq. 4) against exhaustive search.
"""

import itertools
import json
import os
import random

import numpy as np
import pytest

import oracle
from tests import bruteforce

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def fmt_spec(dims):
    """Axis tuples -> spec string in the paper's notation (test-side formatter)."""
    out = []
    for axes in dims:
        if not axes:
            out.append("R")
        elif len(axes) == 1:
            out.append(f"S^{axes[0]}")
        else:
            out.append("S^{" + "".join(str(a) for a in axes) + "}")
    return "".join(out)


def random_dims(rng, ndim, mesh_ndim):
    axes = list(range(mesh_ndim))
    rng.shuffle(axes)
    dims = [[] for _ in range(ndim)]
    for a in axes:
        if rng.random() < 0.7:
            dims[rng.randrange(ndim)].append(a)
    return tuple(tuple(d) for d in dims)


def iota(shape, dtype=np.uint16):
    n = int(np.prod(shape))
    return (np.arange(n, dtype=np.int64) % (1 << (8 * np.dtype(dtype).itemsize))).astype(dtype).reshape(shape)


# ---------------------------------------------------------------- split rule

def test_split_matches_numpy_array_split():
    for length in range(0, 70):
        for k in range(1, 12):
            pieces = np.array_split(np.arange(length), k)
            want = []
            start = 0
            for p in pieces:
                want.append((start, start + len(p)))
                start += len(p)
            assert oracle.split_bounds(length, k) == want, (length, k)


def test_split_uneven_h66_into_4():
    # The U-Transformer skip-tensor workload names the split of H=66 over 4
    # devices as 17,17,16,16.
    assert [hi - lo for lo, hi in oracle.split_bounds(66, 4)] == [17, 17, 16, 16]


# ------------------------------------------------------------- spec parsing

@pytest.mark.parametrize("spec,ndim,mesh_ndim,want", [
    ("S^0RR", 3, 2, ((0,), (), ())),
    ("RS^{01}R", 3, 2, ((), (0, 1), ())),
    ("S_{0}RR", 3, 2, ((0,), (), ())),
    ("RRR", 3, 2, ((), (), ())),
    ("S^{10}R", 2, 2, ((1, 0), ())),
    ("S0 R S1", 3, 2, ((0,), (), (1,))),
    ("R,S^1", 2, 2, ((), (1,))),
])
def test_parse_spec_paper_spellings(spec, ndim, mesh_ndim, want):
    assert oracle.parse_spec(spec, ndim, mesh_ndim) == want


@pytest.mark.parametrize("spec,ndim,mesh_ndim", [
    ("S^0R", 3, 2),       # too few letters
    ("S^0RRR", 3, 2),     # too many
    ("S^2RR", 3, 2),      # axis beyond the mesh
    ("S^0S^0R", 3, 2),    # axis used twice
    ("S^{00}RR", 3, 2),   # axis used twice in one dim
    ("XRR", 3, 2),        # unknown letter
    ("S^RR", 3, 2),       # S without an axis
])
def test_parse_spec_rejects(spec, ndim, mesh_ndim):
    with pytest.raises(ValueError):
        oracle.parse_spec(spec, ndim, mesh_ndim)


# ------------------------------------------------------------------ Fig. 2

def _fig2():
    with open(os.path.join(GOLDEN, "fig2_device_view.json")) as f:
        return json.load(f)


def test_fig2_spec2_replicas_hold_elements_0_to_7():
    g = _fig2()
    x = np.arange(16, dtype=np.int64).reshape(4, 4)
    fact = next(f for f in g["facts"] if f["id"] == "spec2_replica")
    b_ids = g["meshes"]["mesh_B"]["device_ids"]
    shards = oracle.shard(x, (2, 2), g["readings"]["spec2_on_B"])
    for dev in fact["device_ids"]:
        assert sorted(shards[b_ids.index(dev)].ravel().tolist()) == fact["elements"]
    uniq = {tuple(s.ravel().tolist()) for s in shards}
    assert len(uniq) == fact["n_unique_slices"]


@pytest.mark.parametrize("fact_id,src,dst,src_ids,dst_ids", [
    ("task1", "spec1_on_A", "spec2_on_B", "mesh_A", "mesh_B"),
    ("task2", "spec2_on_B", "spec3_on_A", "mesh_B", "mesh_A"),
])
def test_fig2_unit_tasks(fact_id, src, dst, src_ids, dst_ids):
    g = _fig2()
    fact = next(f for f in g["facts"] if f["id"] == fact_id)
    x = np.arange(16, dtype=np.int64).reshape(4, 4)
    tasks = oracle.unit_tasks((4, 4), (2, 2), g["readings"][src], (2, 2), g["readings"][dst])
    assert len(tasks) == fact["n_unit_tasks"]
    first = tasks[0]
    sl = tuple(slice(lo, hi) for lo, hi in first["box"])
    assert x[sl].ravel().tolist() == fact["first_slice_elements"]
    ids = g["meshes"][dst_ids]["device_ids"]
    assert [ids[r] for r in first["receivers"]] == fact["first_receivers"]
    # every unit task is sent from a device that really holds it
    src_shards = oracle.shard(x, (2, 2), g["readings"][src])
    for t in tasks:
        sl = tuple(slice(lo, hi) for lo, hi in t["box"])
        for s in t["senders"]:
            assert set(x[sl].ravel().tolist()) <= set(src_shards[s].ravel().tolist())


# ------------------------------------------------------------------ Table 3

def _table3():
    with open(os.path.join(GOLDEN, "table3_cases.json")) as f:
        return json.load(f)


def test_table3_stated_unit_task_counts():
    g = _table3()
    shape = tuple(g["tensor_shape"])
    stated = [c for c in g["cases"] if "stated_n_unit_tasks" in c]
    assert {c["case"] for c in stated} == {4, 8}
    for c in stated:
        tasks = oracle.unit_tasks(shape, tuple(c["send_mesh"]), c["send_spec"],
                                  tuple(c["recv_mesh"]), c["recv_spec"])
        assert len(tasks) == c["stated_n_unit_tasks"], c["case"]


def test_table3_slices_tile_tensor_and_owners_are_exact():
    # Section 2.2: the unit tasks partition D (their volumes sum to |D|);
    # senders are exactly the owners, receivers exactly the requirers.
    g = _table3()
    shape = (16, 8, 4)  # scaled-down stand-in keeping every split exact or uneven as in the paper
    for c in g["cases"]:
        sm, dm = tuple(c["send_mesh"]), tuple(c["recv_mesh"])
        tasks = oracle.unit_tasks(shape, sm, c["send_spec"], dm, c["recv_spec"])
        cover = np.zeros(shape, dtype=np.int64)
        for t in tasks:
            cover[tuple(slice(lo, hi) for lo, hi in t["box"])] += 1
        assert (cover == 1).all(), c["case"]
        x = iota(shape, np.uint16)
        src = bruteforce.layout(x, sm, oracle.parse_spec(c["send_spec"], 3, 2))
        dst = bruteforce.layout(x, dm, oracle.parse_spec(c["recv_spec"], 3, 2))
        for t in tasks:
            sl = tuple(slice(lo, hi) for lo, hi in t["box"])
            vals = set(x[sl].ravel().tolist())
            owners = [k for k in range(len(src)) if vals <= set(src[k].ravel().tolist())]
            needers = [k for k in range(len(dst)) if vals <= set(dst[k].ravel().tolist())]
            assert t["senders"] == owners, c["case"]
            assert t["receivers"] == needers, c["case"]


def test_table3_naive_case2_sends_everything_from_first_node():
    g = _table3()
    c = next(c for c in g["cases"] if c["case"] == 2)
    tasks = oracle.unit_tasks(tuple(g["tensor_shape"]), tuple(c["send_mesh"]), c["send_spec"],
                              tuple(c["recv_mesh"]), c["recv_spec"])
    node_of = lambda dev: dev // c["send_mesh"][1]  # a mesh row is a node
    assert {node_of(s) for s in oracle.choose_senders_naive(tasks)} == {0}


# --------------------------------------------------------------- brute force

def _brute_cases(n, seed):
    rng = random.Random(seed)
    cases = []
    while len(cases) < n:
        ndim = rng.randint(1, 3)
        shape = tuple(rng.randint(1, 7) for _ in range(ndim))
        smesh = tuple(rng.randint(1, 3) for _ in range(rng.randint(1, 2)))
        dmesh = tuple(rng.randint(1, 3) for _ in range(rng.randint(1, 2)))
        cases.append((shape, smesh, random_dims(rng, ndim, len(smesh)),
                      dmesh, random_dims(rng, ndim, len(dmesh))))
    return cases


@pytest.mark.parametrize("case", _brute_cases(60, 1234))
def test_oracle_matches_brute_force(case):
    shape, smesh, sdims, dmesh, ddims = case
    x = iota(shape, np.uint16)
    src_bf = bruteforce.layout(x, smesh, sdims)
    dst_bf = bruteforce.layout(x, dmesh, ddims)
    sspec, dspec = fmt_spec(sdims), fmt_spec(ddims)
    assert oracle.parse_spec(sspec, len(shape), len(smesh)) == sdims
    for a, b in zip(oracle.shard(x, smesh, sspec), src_bf):
        assert a.shape == b.shape and np.array_equal(a, b)
    out = oracle.reshard(src_bf, shape, smesh, sspec, dmesh, dspec)
    assert len(out) == len(dst_bf)
    for a, b in zip(out, dst_bf):
        assert a.shape == b.shape and np.array_equal(a, b)


def test_brute_force_mesh_order_axis_major():
    # S^{01} on a (2,3) mesh: the shard number is c0*3 + c1 (first listed axis
    # most significant), so device (1,0) = device 3 holds shard 3.
    x = np.arange(6, dtype=np.uint16)
    got = oracle.shard(x, (2, 3), "S^{01}")
    assert [g.tolist() for g in got] == [[0], [1], [2], [3], [4], [5]]
    got = oracle.shard(x, (2, 3), "S^{10}")
    # axes listed (1, 0): shard = c1*2 + c0, device (c0,c1) = (0,1) -> shard 2
    assert [g.tolist() for g in got] == [[0], [2], [4], [1], [3], [5]]


# ---------------------------------------------------------------- invariants

def _fuzz_cases(n, seed, max_len=9):
    rng = random.Random(seed)
    cases = []
    while len(cases) < n:
        ndim = rng.randint(1, 4)
        shape = tuple(rng.randint(0, max_len) if rng.random() < 0.05 else rng.randint(1, max_len)
                      for _ in range(ndim))
        smesh = tuple(rng.randint(1, 4) for _ in range(rng.randint(1, 3)))
        dmesh = tuple(rng.randint(1, 4) for _ in range(rng.randint(1, 3)))
        cases.append((shape, smesh, fmt_spec(random_dims(rng, ndim, len(smesh))),
                      dmesh, fmt_spec(random_dims(rng, ndim, len(dmesh)))))
    return cases


@pytest.mark.parametrize("case", _fuzz_cases(80, 99))
def test_invariants(case):
    shape, sm, ss, dm, ds = case
    x = iota(shape, np.uint32)
    src = oracle.shard(x, sm, ss)
    dst = oracle.reshard(src, shape, sm, ss, dm, ds)
    # I1 reassembly: placing every destination buffer back gives x
    rebuilt = oracle.unshard(dst, shape, dm, ds)
    assert np.array_equal(rebuilt, x)
    # I2 replicas identical: equal boxes carry equal bytes
    ddims = oracle.parse_spec(ds, len(shape), len(dm))
    by_box = {}
    for k, buf in enumerate(dst):
        by_box.setdefault(oracle.device_box(shape, dm, ddims, k), []).append(buf)
    for bufs in by_box.values():
        for b in bufs[1:]:
            assert np.array_equal(b, bufs[0])
    # I4 round trip A -> B -> A
    back = oracle.reshard(dst, shape, dm, ds, sm, ss)
    for a, b in zip(back, src):
        assert np.array_equal(a, b)
    # I5 traffic: unit-task volumes sum to |D|; written = sum of dst shards
    tasks = oracle.unit_tasks(shape, sm, ss, dm, ds)
    vol = sum(int(np.prod([hi - lo for lo, hi in t["box"]])) for t in tasks)
    n = int(np.prod(shape))
    assert vol == n
    rd, wr = oracle.traffic_bytes(shape, 4, dm, ds)
    assert rd == 4 * n and wr == 4 * sum(b.size for b in dst)
    # every receiver of a task gets it, every sender holds it
    sdims = oracle.parse_spec(ss, len(shape), len(sm))
    for t in tasks:
        assert t["senders"] and t["receivers"]
        for s in t["senders"]:
            bx = oracle.device_box(shape, sm, sdims, s)
            assert all(a <= lo and hi <= b for (a, b), (lo, hi) in zip(bx, t["box"]))


@pytest.mark.parametrize("case", _fuzz_cases(25, 7))
def test_identity_reshard_is_copy(case):
    shape, sm, ss, _, _ = case
    x = iota(shape, np.uint16)
    src = oracle.shard(x, sm, ss)
    out = oracle.reshard(src, shape, sm, ss, sm, ss)
    for a, b in zip(out, src):
        assert np.array_equal(a, b)
        assert a is not b


@pytest.mark.parametrize("seed", range(20))
def test_composition(seed):
    rng = random.Random(seed)
    ndim = rng.randint(1, 3)
    shape = tuple(rng.randint(1, 8) for _ in range(ndim))
    meshes = [tuple(rng.randint(1, 3) for _ in range(rng.randint(1, 2))) for _ in range(3)]
    specs = [fmt_spec(random_dims(rng, ndim, len(m))) for m in meshes]
    x = iota(shape, np.uint16)
    a = oracle.shard(x, meshes[0], specs[0])
    b = oracle.reshard(a, shape, meshes[0], specs[0], meshes[1], specs[1])
    c1 = oracle.reshard(b, shape, meshes[1], specs[1], meshes[2], specs[2])
    c2 = oracle.reshard(a, shape, meshes[0], specs[0], meshes[2], specs[2])
    for u, v in zip(c1, c2):
        assert np.array_equal(u, v)


def test_special_cases():
    x = iota((6, 5), np.uint16)
    # to a fully replicated layout is an all-gather: every buffer is x
    src = oracle.shard(x, (2, 2), "S^0S^1")
    for buf in oracle.reshard(src, (6, 5), (2, 2), "S^0S^1", (3,), "RR"):
        assert np.array_equal(buf, x)
    # from fully replicated to sharded is plain slicing
    src = oracle.shard(x, (2,), "RR")
    out = oracle.reshard(src, (6, 5), (2,), "RR", (3,), "S^0R")
    assert [b.tolist() for b in out] == [x[0:2].tolist(), x[2:4].tolist(), x[4:6].tolist()]


def test_raw_bits_survive():
    # NaN payloads and -0.0 must pass through bit for bit.
    bits = np.array([0x7E01, 0xFE02, 0x8000, 0x7C00, 0xFC00, 0x0001, 0x7FFF, 0xFFFF], dtype=np.uint16)
    x = bits.view(np.float16).reshape(2, 4)
    src = oracle.shard(x, (2,), "S^0R")
    out = oracle.reshard(src, (2, 4), (2,), "S^0R", (2,), "RS^0")
    assert out[0].dtype == np.float16
    got = np.concatenate([o.view(np.uint16) for o in out], axis=1)
    assert np.array_equal(got, bits.reshape(2, 4))


def test_unshard_rejects_inconsistent_replicas():
    x = iota((4,), np.uint16)
    src = oracle.shard(x, (2,), "R")
    src[1] = src[1].copy()
    src[1][0] ^= 1
    with pytest.raises(ValueError):
        oracle.unshard(src, (4,), (2,), "R")


# ----------------------------------------------------------- sender choice

def _makespan(tasks, chosen, n, itemsize=1):
    load = [0] * n
    for t, s in zip(tasks, chosen):
        load[s] += int(np.prod([hi - lo for lo, hi in t["box"]])) * itemsize
    return max(load)


def _optimum(tasks, n):
    best = None
    for choice in itertools.product(*[t["senders"] for t in tasks]):
        m = _makespan(tasks, choice, n)
        best = m if best is None or m < best else best
    return best


def _synthetic_tasks(sizes, senders):
    return [{"box": ((0, s),), "senders": list(c), "receivers": [0]} for s, c in zip(sizes, senders)]


@pytest.mark.parametrize("seed", range(40))
def test_lpt_within_graham_bound_identical_senders(seed):
    # Eq. 4 with every sender eligible is makespan scheduling on identical
    # machines; greedy longest-first is within 4/3 - 1/(3m) of the optimum.
    rng = random.Random(seed)
    m = rng.randint(2, 4)
    sizes = [rng.randint(1, 20) for _ in range(rng.randint(2, 7))]
    tasks = _synthetic_tasks(sizes, [range(m)] * len(sizes))
    got = _makespan(tasks, oracle.choose_senders_lpt(tasks, 1, m), m)
    opt = _optimum(tasks, m)
    assert got * 3 * m <= opt * (4 * m - 1)


def test_lpt_sorts_longest_first():
    # sizes 1,1,2 on two senders: longest-first reaches the optimum 2;
    # visiting in the given order would give 3.
    tasks = _synthetic_tasks([1, 1, 2], [[0, 1]] * 3)
    assert _makespan(tasks, oracle.choose_senders_lpt(tasks, 1, 2), 2) == 2


def test_lpt_optimal_on_table3_cases():
    # The paper's tasks are even slices, where greedy balancing is optimal.
    g = _table3()
    for c in g["cases"]:
        sm = tuple(c["send_mesh"])
        tasks = oracle.unit_tasks((16, 8, 4), sm, c["send_spec"], tuple(c["recv_mesh"]), c["recv_spec"])
        if np.prod([len(t["senders"]) for t in tasks]) > 50000:
            continue
        n = int(np.prod(sm))
        got = _makespan(tasks, oracle.choose_senders_lpt(tasks, 2, n), n, 2)
        assert got == 2 * _optimum(tasks, n), c["case"]


def test_naive_picks_lowest_index():
    tasks = _synthetic_tasks([5, 3], [[2, 1, 3], [4, 0]])
    assert oracle.choose_senders_naive(tasks) == [1, 0]


# ------------------------------------------------- permuted local layouts

def _perm_cases(n, seed):
    rng = random.Random(seed)
    out = []
    for shape, smesh, sdims, dmesh, ddims in _brute_cases(n, seed):
        sp = list(range(len(shape)))
        dp = list(range(len(shape)))
        rng.shuffle(sp)
        rng.shuffle(dp)
        out.append((shape, smesh, sdims, tuple(sp), dmesh, ddims, tuple(dp)))
    return out


@pytest.mark.parametrize("case", _perm_cases(40, 4321))
def test_permuted_layouts_match_brute_force(case):
    # the element-by-element formulation places each element at its rank
    # inside the shard, read in the buffer's dimension order
    shape, smesh, sdims, sp, dmesh, ddims, dp = case
    x = iota(shape, np.uint16)
    src_bf = bruteforce.layout(x, smesh, sdims, sp)
    dst_bf = bruteforce.layout(x, dmesh, ddims, dp)
    sspec, dspec = fmt_spec(sdims), fmt_spec(ddims)
    for d, (a, b) in enumerate(zip(oracle.shard(x, smesh, sspec, sp), src_bf)):
        assert a.shape == b.shape == oracle.local_shape(shape, smesh, sspec, d, sp) and np.array_equal(a, b)
    out = oracle.reshard(src_bf, shape, smesh, sspec, dmesh, dspec, src_perm=sp, dst_perm=dp)
    for a, b in zip(out, dst_bf):
        assert a.shape == b.shape and np.array_equal(a, b)


def test_permuted_layout_special_cases():
    x = iota((5, 7), np.uint32)
    # one device, both dimensions kept whole: the buffer is the textbook transpose
    (t,) = oracle.shard(x, (1,), "RR", (1, 0))
    assert t.shape == (7, 5) and all(t[j, i] == x[i, j] for i in range(5) for j in range(7))
    # moving a tensor from the plain layout to the transposed one and back
    there = oracle.reshard(oracle.shard(x, (2,), "S^0R"), (5, 7), (2,), "S^0R", (3,), "RS^0", dst_perm=(1, 0))
    assert [a.shape for a in there] == [(3, 5), (2, 5), (2, 5)]
    back = oracle.reshard(there, (5, 7), (3,), "RS^0", (2,), "S^0R", src_perm=(1, 0))
    for a, b in zip(back, oracle.shard(x, (2,), "S^0R")):
        assert np.array_equal(a, b)
    # the identity permutation is the plain layout
    for a, b in zip(oracle.shard(x, (2,), "S^0R", (0, 1)), oracle.shard(x, (2,), "S^0R")):
        assert np.array_equal(a, b)
    with pytest.raises(ValueError):
        oracle.shard(x, (2,), "S^0R", (0, 0))
    with pytest.raises(ValueError):
        oracle.shard(x, (2,), "S^0R", (0, 1, 2))
