"""C-ABI checks that need no GPU: exports, planning, errors, host interpreter.

The planner's unit tasks, senders, local shapes and traffic totals are
compared exactly with the oracle; the descriptor table is run on host
memory by reshard_debug_execute_host and compared bit for bit with the
oracle's destination shards (guard bytes around every buffer must stay
untouched).  No kernel runs here.
"""

import ctypes
import os
import random
import re

import numpy as np
import pytest

import oracle
from paper_2211_05322_amd import binding as B
from paper_2211_05322_amd.workloads import WORKLOADS
from tests.test_oracle_pins import fmt_spec, random_dims

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "reshard.h")

_NP = {"float16": np.float16, "float32": np.float32, "uint8": np.uint8, "float64": np.float64,
       "int16": np.int16, "int32": np.int32, "int64": np.int64, "bfloat16": np.uint16}


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(reshard_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = B.load()
    names = declared_functions()
    assert {"reshard_plan", "reshard_execute", "reshard_plan_destroy", "reshard_plan_local_shape",
            "reshard_plan_stats", "reshard_last_error"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n
    assert B.reshard_version() == "0.1.0"


def plan_of(shape, dtype, sm, ss, dm, ds, **kw):
    return B.reshard_plan(shape, dtype, sm, ss, dm, ds, **kw)


def check_against_oracle(shape, dtype, sm, ss, dm, ds, flags=0, itemsize=None):
    p = plan_of(shape, dtype, sm, ss, dm, ds, flags=flags)
    es = itemsize or np.dtype(_NP[dtype]).itemsize
    tasks = oracle.unit_tasks(shape, sm, ss, dm, ds)
    st = B.reshard_plan_stats(p)
    assert st["n_unit_tasks"] == len(tasks)
    rd, wr = oracle.traffic_bytes(shape, es, dm, ds)
    assert (st["bytes_read"], st["bytes_written"]) == (rd, wr)
    if flags & B.RESHARD_SENDER_NAIVE:
        chosen = oracle.choose_senders_naive(tasks)
    else:
        chosen = oracle.choose_senders_lpt(tasks, es, int(np.prod(sm)))
    for i, t in enumerate(tasks):
        got = B.reshard_plan_unit_task(p, i)
        assert got["box"] == t["box"]
        assert got["senders"] == t["senders"]
        assert got["receivers"] == t["receivers"]
        assert got["sender"] == chosen[i]
    for side, mesh, spec in ((0, sm, ss), (1, dm, ds)):
        for k in range(int(np.prod(mesh))):
            assert B.reshard_plan_local_shape(p, side, k) == oracle.local_shape(shape, mesh, spec, k)
    return p


# ----------------------------------------------------------------- planning

def test_fig2_plans():
    check_against_oracle((4, 4), "float32", (2, 2), "S^{01}R", (2, 2), "S^0R")
    check_against_oracle((4, 4), "float32", (2, 2), "S^0R", (2, 2), "S^0R")


@pytest.mark.parametrize("case", range(1, 10))
@pytest.mark.parametrize("flags", [0, B.RESHARD_SENDER_NAIVE])
def test_table3_plans_full_size(case, flags):
    import json
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "table3_cases.json")))
    c = g["cases"][case - 1]
    check_against_oracle(tuple(g["tensor_shape"]), "float16", tuple(c["send_mesh"]), c["send_spec"],
                         tuple(c["recv_mesh"]), c["recv_spec"], flags=flags)


@pytest.mark.parametrize("wid", sorted(WORKLOADS))
def test_workload_plans(wid):
    w = WORKLOADS[wid]
    p = check_against_oracle(w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec)
    st = B.reshard_plan_stats(p)
    assert B.reshard_plan_alignment(p) == 16  # every workload takes the 16-byte path
    assert st["max_fanout"] == {1: 2, 2: 1, 3: 8, 4: 2, 5: 4}[wid]


def _fuzz(n, seed, max_len=12):
    rng = random.Random(seed)
    out = []
    while len(out) < n:
        ndim = rng.randint(1, 5)
        shape = tuple(rng.randint(0, max_len) if rng.random() < 0.05 else rng.randint(1, max_len)
                      for _ in range(ndim))
        sm = tuple(rng.randint(1, 4) for _ in range(rng.randint(1, 3)))
        dm = tuple(rng.randint(1, 4) for _ in range(rng.randint(1, 3)))
        out.append((shape, rng.choice(["uint8", "float16", "float32", "float64"]), sm,
                    fmt_spec(random_dims(rng, ndim, len(sm))), dm, fmt_spec(random_dims(rng, ndim, len(dm))),
                    rng.choice([0, 0, B.RESHARD_SENDER_NAIVE, B.RESHARD_TASK_ORDER,
                                B.RESHARD_XCD_REMAP | B.RESHARD_SENDER_NAIVE])))
    return out


@pytest.mark.parametrize("case", _fuzz(60, 5))
def test_fuzz_plans(case):
    shape, dt, sm, ss, dm, ds, flags = case
    check_against_oracle(shape, dt, sm, ss, dm, ds, flags=flags)


# -------------------------------------------------------- host interpreter

GUARD = 64


def run_host(p, src_arrays, dst_shapes, np_dtype):
    """Execute the descriptor table on host buffers with guard bands."""
    es = np.dtype(np_dtype).itemsize
    srcs = []
    for a in src_arrays:
        raw = np.full(a.nbytes + 2 * GUARD, 0xA5, dtype=np.uint8)
        raw[GUARD:GUARD + a.nbytes] = np.ascontiguousarray(a).view(np.uint8).ravel()
        srcs.append(raw)
    dsts = [np.full(int(np.prod(s)) * es + 2 * GUARD, 0x5A, dtype=np.uint8) for s in dst_shapes]
    # 16-byte aligned views one guard band in
    sp = [r.ctypes.data + GUARD if r.size > 2 * GUARD else None for r in srcs]
    dp = [r.ctypes.data + GUARD if r.size > 2 * GUARD else None for r in dsts]
    for q in sp + dp:
        assert q is None or q % 16 == 0
    B._check(B.load().reshard_debug_execute_host(p.handle, B._ptrs(sp), B._ptrs(dp)))
    outs = []
    for r, s in zip(dsts, dst_shapes):
        assert (r[:GUARD] == 0x5A).all() and (r[r.size - GUARD:] == 0x5A).all(), "write outside buffer"
        outs.append(r[GUARD:r.size - GUARD].view(np_dtype).reshape(s))
    for r, a in zip(srcs, src_arrays):
        assert (r[GUARD:GUARD + a.nbytes] == np.ascontiguousarray(a).view(np.uint8).ravel()).all()
    return outs


def host_case(shape, dt, sm, ss, dm, ds, flags=0, seed=0, **kw):
    np_dtype = _NP[dt]
    es = np.dtype(np_dtype).itemsize
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 256, size=int(np.prod(shape)) * es, dtype=np.uint8).view(np_dtype).reshape(shape)
    src = oracle.shard(x, sm, ss)
    want = oracle.reshard(src, shape, sm, ss, dm, ds)
    p = plan_of(shape, dt, sm, ss, dm, ds, flags=flags, **kw)
    got = run_host(p, src, [w.shape for w in want], np_dtype)
    for g, w in zip(got, want):
        assert g.shape == w.shape
        assert np.array_equal(g.view(f"u{es}"), w.view(f"u{es}"))


@pytest.mark.parametrize("case", _fuzz(80, 11))
def test_host_interpreter_fuzz(case):
    shape, dt, sm, ss, dm, ds, flags = case
    host_case(shape, dt, sm, ss, dm, ds, flags)


def _fuzz_lowering(n, seed):
    """Random tensors with longer rows (so every chunk kind occurs), random
    meshes and specs, crossed with random lowering flags and tunings."""
    rng = random.Random(seed)
    flag_sets = [0, B.RESHARD_NO_GATHER, B.RESHARD_LDS_STAGING, B.RESHARD_NO_REALIGN | B.RESHARD_NO_GATHER,
                 B.RESHARD_XCD_REMAP, B.RESHARD_TASK_ORDER | B.RESHARD_SENDER_NAIVE,
                 B.RESHARD_STRATEGY_SENDRECV, B.RESHARD_STRATEGY_ALLGATHER]
    out = []
    while len(out) < n:
        ndim = rng.randint(1, 4)
        shape = tuple(rng.randint(1, 9) for _ in range(ndim - 1)) + (rng.randint(16, 700),)
        sm = tuple(rng.randint(1, 4) for _ in range(rng.randint(1, 3)))
        dm = tuple(rng.randint(1, 4) for _ in range(rng.randint(1, 3)))
        kw = {"flags": rng.choice(flag_sets)}
        if rng.random() < 0.7:
            kw["chunk_bytes"] = rng.choice([64, 256, 1000, 4096, 20000])
            kw["block_threads"] = rng.choice([64, 128, 256, 512, 1024])
            kw["max_wgs_per_cu"] = rng.choice([0, -1, 2, 5])
            kw["gather_band"] = rng.choice([0, 0, 1, 3])
        out.append((shape, rng.choice(["uint8", "float16", "float32", "float64"]), sm,
                    fmt_spec(random_dims(rng, ndim, len(sm))), dm, fmt_spec(random_dims(rng, ndim, len(dm))), kw))
    return out


@pytest.mark.parametrize("case", _fuzz_lowering(400, 2024))
def test_host_lowering_fuzz(case):
    """The GPU lowering fuzz's cases (every chunk kind, random flags and
    tunings) through the host interpreter against the oracle."""
    shape, dt, sm, ss, dm, ds, kw = case
    kw = dict(kw)
    flags = kw.pop("flags", 0)
    host_case(shape, dt, sm, ss, dm, ds, flags, **kw)


@pytest.mark.parametrize("chunk", [0, 16, 48, 1000, 4096])
@pytest.mark.parametrize("case", _fuzz(12, 23, max_len=40))
def test_host_interpreter_chunking(case, chunk):
    shape, dt, sm, ss, dm, ds, flags = case
    host_case(shape, dt, sm, ss, dm, ds, flags, chunk_bytes=chunk)


@pytest.mark.parametrize("wid", sorted(WORKLOADS))
def test_host_interpreter_scaled_workloads(wid):
    # the workload's meshes and specs on a shrunken tensor (every dim cut so
    # splits stay exact or uneven as in the original)
    w = WORKLOADS[wid]
    small = {1: (64, 96), 2: (4, 64, 96), 3: (2, 24, 200), 4: (4, 8, 66, 16), 5: (2, 64, 384)}[wid]
    host_case(small, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec)


def test_host_interpreter_misaligned_phase_and_long_runs():
    # fp16 rows of odd length: source and destination 16-byte phases differ
    host_case((3, 37, 29), "float16", (2, 2), "S^0S^1R", (3,), "RRS^0")
    # long contiguous runs with a ragged tail
    host_case((5, 1000), "float16", (1,), "RR", (2,), "RS^0")
    # > 3 non-collapsible outer levels
    host_case((3, 4, 3, 4, 3, 8), "uint8", (2, 2, 2), "RS^0RS^1RS^2", (2, 2), "S^0RS^1RRR")


# ------------------------------------------------- LDS realignment path

REALIGN_CASES = [
    # (shape, dtype, src mesh, src spec, dst mesh, dst spec): rows whose source
    # and destination 16-byte phases differ
    ((3, 37, 290), "float16", (2, 2), "S^0S^1R", (3,), "RRS^0"),       # odd rows, many phases
    ((6, 4000), "float16", (3,), "RS^0", (2,), "RS^0"),                 # long rows, 1 dst phase shift
    ((5, 1000), "uint8", (1,), "RR", (3,), "RS^0"),                     # fan-out 1, byte rows
    ((4, 96, 70), "float16", (2,), "S^0RR", (2, 2), "RS^0S^1"),         # strides not multiples of 16
    ((2, 8, 3, 333), "float32", (2, 2), "RS^0RS^1", (3,), "RRRS^0"),    # 3 outer levels
    ((7, 130), "float64", (2,), "S^0R", (3, 2), "RS^0"),                # fan-out 2 (replicated over axis 1)
    ((2, 9000), "float16", (1,), "RR", (2,), "RS^0"),                   # rows longer than one segment
]


@pytest.mark.parametrize("case", REALIGN_CASES)
@pytest.mark.parametrize("chunk", [0, 100, 5000])
def test_host_realign_path(case, chunk):
    shape, dt, sm, ss, dm, ds = case
    ng = B.RESHARD_NO_GATHER  # some cases take the unaligned row gather by default
    p = plan_of(shape, dt, sm, ss, dm, ds, chunk_bytes=chunk, flags=ng)
    assert B.reshard_plan_realign_chunks(p) > 0, "case should take the realignment path"
    assert B.reshard_plan_lds_bytes(p) == 0
    host_case(shape, dt, sm, ss, dm, ds, chunk_bytes=chunk, flags=ng)
    host_case(shape, dt, sm, ss, dm, ds, chunk_bytes=chunk)
    q = plan_of(shape, dt, sm, ss, dm, ds, flags=B.RESHARD_NO_REALIGN | ng)
    assert B.reshard_plan_realign_chunks(q) == 0
    host_case(shape, dt, sm, ss, dm, ds, flags=B.RESHARD_NO_REALIGN | ng)
    r = plan_of(shape, dt, sm, ss, dm, ds, flags=B.RESHARD_LDS_STAGING | ng)
    assert B.reshard_plan_lds_bytes(r) > 0
    host_case(shape, dt, sm, ss, dm, ds, flags=B.RESHARD_LDS_STAGING | ng, chunk_bytes=chunk)


# Row groups whose destination rows are contiguous only in runs -- the
# source split along a middle dimension, the destination along an outer one
# -- with rows in different 16-byte phases: one unaligned-gather region per
# run when every run holds at least a chunk, else the realignment path.
RUN_CASES = [
    ((4, 130, 101), "uint8", (2,), "R S^0 R", (2,), "S^0 R R"),
    ((6, 130, 203), "uint8", (2,), "R S^0 R", (3,), "S^0 R R"),
    ((4, 66, 130, 45), "uint8", (2, 2), "R S^0 S^1 R", (2,), "S^0 R R R"),   # runs over two levels
    ((4, 41, 77), "float16", (2, 2), "R S^0 S^1", (2,), "S^0 R R"),          # two segments per row
    ((10, 33, 150), "float32", (2,), "R S^0 R", (5, 2), "S^0 R R"),          # fan-out 2
    ((4, 41, 77), "float16", (2, 2), "R S^0 S^1", (2, 3), "S^0 R R"),        # fan-out 3
]


@pytest.mark.parametrize("case", RUN_CASES)
@pytest.mark.parametrize("chunk", [0, 256, 1024])
def test_host_unaligned_gather_in_runs(case, chunk):
    p = plan_of(*case, chunk_bytes=chunk)
    if chunk:
        assert B.reshard_plan_unaligned_gather_chunks(p) > 0 and B.reshard_plan_realign_chunks(p) == 0
    host_case(*case, chunk_bytes=chunk)


def test_short_runs():
    # runs of 21 or 20 rows x 154 bytes (about 3 KiB, shorter than the
    # automatic 4 KiB chunk) take the unaligned row gather, one short chunk
    # per run; runs of 6 or 5 rows (under 1 KiB) keep the realignment path
    p = plan_of((4, 41, 77), "float16", (2, 2), "R S^0 S^1", (2,), "S^0 R R")
    assert B.reshard_plan_unaligned_gather_chunks(p) > 0 and B.reshard_plan_realign_chunks(p) == 0
    host_case((4, 41, 77), "float16", (2, 2), "R S^0 S^1", (2,), "S^0 R R")
    p = plan_of((4, 11, 77), "float16", (2, 2), "R S^0 S^1", (2,), "S^0 R R")
    assert B.reshard_plan_unaligned_gather_chunks(p) == 0 and B.reshard_plan_realign_chunks(p) > 0
    host_case((4, 11, 77), "float16", (2, 2), "R S^0 S^1", (2,), "S^0 R R")


def test_aligned_workloads_do_not_realign():
    for w in WORKLOADS.values():
        p = plan_of(w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec)
        assert B.reshard_plan_realign_chunks(p) == 0
        assert B.reshard_plan_lds_bytes(p) == 0


# ------------------------------------------------------------------ errors

@pytest.mark.parametrize("args,status", [
    (((4, 4), "float32", (2, 2), "S^0", (2, 2), "RR"), B.RESHARD_EINVAL),          # spec too short
    (((4, 4), "float32", (2, 2), "S^2R", (2, 2), "RR"), B.RESHARD_EINVAL),         # axis outside mesh
    (((4, 4), "float32", (2, 2), "S^0S^0", (2, 2), "RR"), B.RESHARD_EINVAL),       # axis reused
    (((4, 4), "float32", (2, 2), "Q R", (2, 2), "RR"), B.RESHARD_EINVAL),          # bad letter
    (((4, 4), "float32", (2, 2), "S^{0R", (2, 2), "RR"), B.RESHARD_EINVAL),        # missing brace
    (((4, -1), "float32", (2, 2), "RR", (2, 2), "RR"), B.RESHARD_EINVAL),          # negative dim
    (((4, 4), "float32", (2, 0), "RR", (2, 2), "RR"), B.RESHARD_EINVAL),           # empty mesh axis
    (((4, 4), "float32", (16, 16), "RR", (16, 16), "RR"), B.RESHARD_EUNSUPPORTED),  # 512 buffers
])
def test_plan_errors(args, status):
    with pytest.raises(B.ReshardError) as e:
        plan_of(*args)
    assert e.value.status == status
    assert B.reshard_last_error()


def test_plan_error_ndim_and_nulls():
    lib = B.load()
    h = ctypes.c_void_p()
    shape = B._i64([2, 2])
    mesh = B._i64([2])
    assert lib.reshard_plan(0, shape, 2, 1, mesh, b"", 1, mesh, b"", 0, ctypes.byref(h)) == B.RESHARD_EINVAL
    assert lib.reshard_plan(9, shape, 2, 1, mesh, b"R" * 9, 1, mesh, b"R" * 9, 0,
                            ctypes.byref(h)) == B.RESHARD_EINVAL
    assert lib.reshard_plan(2, None, 2, 1, mesh, b"RR", 1, mesh, b"RR", 0, ctypes.byref(h)) == B.RESHARD_EINVAL
    assert lib.reshard_plan(2, shape, 2, 1, mesh, None, 1, mesh, b"RR", 0, ctypes.byref(h)) == B.RESHARD_EINVAL
    assert lib.reshard_plan(2, shape, 2, 1, mesh, b"RR", 1, mesh, b"RR", 0, None) == B.RESHARD_EINVAL
    assert lib.reshard_plan(2, shape, 99, 1, mesh, b"RR", 1, mesh, b"RR", 0, ctypes.byref(h)) == B.RESHARD_EINVAL
    assert lib.reshard_plan(2, shape, 2, 1, mesh, b"RR", 1, mesh, b"RR", 0x80, ctypes.byref(h)) == B.RESHARD_EINVAL
    assert lib.reshard_plan(2, shape, 2, 0, mesh, b"RR", 1, mesh, b"RR", 0, ctypes.byref(h)) == B.RESHARD_EINVAL
    assert "1..8" in B.reshard_last_error()
    lib.reshard_plan_destroy(None)  # NULL accepted
    assert lib.reshard_execute(None, None, None, None) == B.RESHARD_EINVAL
    assert lib.reshard_plan_upload(None) == B.RESHARD_EINVAL
    # a plan with nothing to move has no table: uploading it touches no device
    empty = plan_of((0, 4), "float16", (2,), "S^0R", (2,), "RS^0")
    assert lib.reshard_plan_upload(empty.handle) == B.RESHARD_OK


def test_default_chunking_scales_past_the_chunk_limit():
    # 300 GiB of unique bytes: 16 KiB chunks would exceed the 2^24-chunk
    # table; automatic chunking grows instead (plan only, no data)
    p = plan_of((300 << 30,), "uint8", (1,), "R", (2,), "S^0")
    st = B.reshard_plan_stats(p)
    assert st["bytes_read"] == 300 << 30
    assert st["n_descriptors"] <= 1 << 22
    # an explicitly tiny chunk on a large tensor is refused, not truncated
    with pytest.raises(B.ReshardError) as e:
        plan_of((1 << 33,), "uint8", (1,), "R", (1,), "R", chunk_bytes=256)
    assert e.value.status == B.RESHARD_EUNSUPPORTED and "2^24" in str(e.value)


def test_query_errors():
    p = plan_of((4, 4), "float16", (2,), "S^0R", (2,), "RS^0")
    lib = B.load()
    out = (ctypes.c_int64 * 2)()
    assert lib.reshard_plan_local_shape(p.handle, 2, 0, out) == B.RESHARD_EINVAL
    assert lib.reshard_plan_local_shape(p.handle, 0, 5, out) == B.RESHARD_EINVAL
    assert lib.reshard_plan_unit_task(p.handle, 99, out, out, None, None, 0, None, None, 0, None) == B.RESHARD_EINVAL
    with pytest.raises(B.ReshardError):
        B.reshard_plan((4, 4), "float16", (2,), "RR", (2,), "RR", block_threads=100)
    for cap in (1, 33, -2):
        with pytest.raises(B.ReshardError):
            B.reshard_plan((4, 4), "float16", (2,), "RR", (2,), "RR", max_wgs_per_cu=cap)
    with pytest.raises(B.ReshardError):
        B.reshard_plan((4, 4), "float16", (2,), "RR", (2,), "RR", gather_band=-1)


def test_execute_rejects_null_buffer_on_host_interpreter():
    p = plan_of((4, 4), "float16", (2,), "S^0R", (2,), "RS^0")
    a = np.zeros((2, 4), np.float16)
    with pytest.raises(B.ReshardError):
        B.reshard_debug_execute_host(p, [a, None], [np.zeros((4, 2), np.float16)] * 2)


def test_empty_tensor_and_empty_shards():
    # zero-size tensor: no tasks, nothing to do
    p = plan_of((0, 4), "float32", (2,), "S^0R", (2,), "RS^0")
    st = B.reshard_plan_stats(p)
    assert st["n_unit_tasks"] == 0 and st["n_descriptors"] == 0
    B.reshard_debug_execute_host(p, [None, None], [None, None])
    # 3 rows over 4 devices: the last shard is empty and may be NULL
    host_case((3, 8), "float32", (4,), "S^0R", (2,), "RS^0")
    p = plan_of((3, 8), "float32", (4,), "S^0R", (2,), "RS^0")
    assert B.reshard_plan_local_shape(p, 0, 3) == (0, 8)


# ------------------------------------------ comparison strategies (f2)

@pytest.mark.parametrize("strategy", [B.RESHARD_STRATEGY_SENDRECV, B.RESHARD_STRATEGY_ALLGATHER])
@pytest.mark.parametrize("case", _fuzz(30, 31))
def test_host_strategies_fuzz(strategy, case):
    shape, dt, sm, ss, dm, ds, flags = case
    host_case(shape, dt, sm, ss, dm, ds, flags | strategy)


@pytest.mark.parametrize("strategy", [B.RESHARD_STRATEGY_SENDRECV, B.RESHARD_STRATEGY_ALLGATHER])
def test_strategy_traffic(strategy):
    # both comparison strategies read every slice once per receiver
    for w in WORKLOADS.values():
        b = B.reshard_plan_stats(plan_of(w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec))
        s = B.reshard_plan_stats(plan_of(w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec,
                                         flags=strategy))
        assert s["bytes_written"] == b["bytes_written"]
        assert s["bytes_read"] == b["bytes_written"]  # R x |D| (every slice has R receivers)


def test_strategy_flags_exclusive():
    with pytest.raises(B.ReshardError):
        plan_of((4, 4), "float16", (2,), "RR", (2,), "RR",
                flags=B.RESHARD_STRATEGY_SENDRECV | B.RESHARD_STRATEGY_ALLGATHER)


# ------------------------------------------------------------ row gather

GATHER_CASES = [
    ((8, 64, 1024), "float16", (2, 4), "RRS^{01}", (2, 4), "RS^0R"),
    ((3, 40, 640), "float32", (1, 4), "RRS^1", (2,), "RRR"),
    ((6, 8, 10, 256), "float16", (2, 2), "RRRS^{01}", (3,), "RS^0RR"),
    ((16, 4, 96), "float64", (3,), "RRS^0", (2, 2), "S^0RR"),
    ((2, 64, 1024), "float16", (4, 8), "RRS^{01}", (4, 8), "RS^1R"),
    ((2, 8, 640), "float16", (1, 4), "RRS^1", (3, 4), "RRR"),                # fan-out 12: runtime receiver loop
]


@pytest.mark.parametrize("case", GATHER_CASES)
@pytest.mark.parametrize("chunk", [0, 256, 3000])
@pytest.mark.parametrize("band", [0, 1, 3])
def test_host_gather(case, chunk, band):
    shape, dt, sm, ss, dm, ds = case
    p = plan_of(shape, dt, sm, ss, dm, ds, chunk_bytes=chunk, gather_band=band)
    assert B.reshard_plan_gather_chunks(p) > 0, "case should take the row-gather path"
    host_case(shape, dt, sm, ss, dm, ds, chunk_bytes=chunk, gather_band=band)
    q = plan_of(shape, dt, sm, ss, dm, ds, flags=B.RESHARD_NO_GATHER)
    assert B.reshard_plan_gather_chunks(q) == 0
    host_case(shape, dt, sm, ss, dm, ds, flags=B.RESHARD_NO_GATHER)


@pytest.mark.parametrize("shape", [(2, 64, 512), (4, 96, 768), (3, 50, 1024)])
def test_gather_tail_halves_parity(shape):
    # automatic chunk sizes cut the last fifth of the row-gather chunks in
    # halves; the halves' origins come from the descriptor arithmetic,
    # checked against the oracle through the host interpreter
    args = (shape, "float16", (4, 8), "RRS^{01}", (4, 8), "RS^1R")
    assert B.reshard_plan_gather_chunks(plan_of(*args)) > 0
    host_case(*args)


@pytest.mark.parametrize("band", [1, 3, 5])
def test_gather_tail_halves_with_bands(band):
    # column bands change the slot -> offset arithmetic the halves rely on
    args = ((3, 64, 1024), "float16", (4, 8), "RRS^{01}", (4, 8), "RS^1R")
    assert B.reshard_plan_gather_chunks(plan_of(*args, gather_band=band)) > 0
    host_case(*args, gather_band=band)


@pytest.mark.parametrize("wid", [3, 5])
def test_gather_tail_halves_count(wid):
    # at full size the automatic chunk is 16 KiB: the last fifth of the
    # chunks become two each; an explicit chunk size keeps every chunk whole
    w = WORKLOADS[wid]
    args = (w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec)
    whole = B.reshard_plan_gather_chunks(plan_of(*args, chunk_bytes=16384))
    assert whole == w.numel * w.itemsize // 16384
    assert B.reshard_plan_gather_chunks(plan_of(*args)) == whole + whole // 5


def test_gather_band_chunk_count():
    # bands tile the rows: same slots in total, each band's chunks separate
    shape, dt, sm, ss, dm, ds = GATHER_CASES[4]
    es = 2
    row_slots = shape[2] * es // 16
    rows = shape[0] * shape[1] // 8
    for band, cb in ((0, 4096), (1, 4096), (4, 4096), (5, 1024), (32, 4096), (40, 4096)):
        p = plan_of(shape, dt, sm, ss, dm, ds, chunk_bytes=cb, gather_band=band)
        nseg = 32
        b = band if 0 < band < nseg else nseg
        per_row = [min(b, nseg - b0) * row_slots // nseg for b0 in range(0, nseg, b)]
        want = 8 * sum(-(-rows * w // (cb // 16)) for w in per_row)
        assert B.reshard_plan_gather_chunks(p) == want, band


# ------------------------------------------------ unaligned row gather

UNALIGNED_GATHER_CASES = [
    # segments of any width >= 16 bytes, any 16-byte phase, contiguous destination rows
    ((2, 64, 12300), "float16", (4, 8), "RRS^{01}", (4, 8), "RS^1R"),  # 770/768-byte segments, 24600-byte rows
    ((6, 4000), "float16", (3,), "RS^0", (2,), "RS^0"),                 # uneven cut of 2000 by 1334
    ((4, 32, 1000), "float16", (1, 4), "RRS^1", (2,), "RRR"),           # 500-byte segments, fan-out 2
    ((3, 10, 7, 333), "float32", (2, 3), "RRRS^{01}", (3,), "S^0RRR"),  # 6 senders of 222/220 bytes
    ((5, 1000), "uint8", (4,), "RS^0", (1,), "RR"),                     # byte elements, 250-byte segments
    ((2, 5, 8, 12), "float64", (2, 2), "RRRS^{01}", (2,), "RRRR"),      # 24-byte segments
    ((2, 8, 650), "float16", (1, 4), "RRS^1", (3, 4), "RRR"),           # fan-out 12: runtime receiver loop
    ((3, 16, 1000), "uint8", (5,), "RRS^0", (2, 5), "RRR"),             # fan-out 10, 200-byte segments
    # one sender per row, the two sides' rows in different 16-byte phases
    ((8, 64, 1230), "float16", (1,), "RRR", (4,), "RRS^0"),             # 616/614-byte rows from one source
    ((7, 130), "float64", (2,), "S^0R", (3, 2), "RS^0"),                # fan-out 2, 344/352-byte rows
    ((5, 1000), "uint8", (1,), "RR", (3,), "RS^0"),                     # byte rows of 334/333
]


@pytest.mark.parametrize("case", UNALIGNED_GATHER_CASES)
@pytest.mark.parametrize("chunk", [0, 64, 3000])
def test_host_unaligned_gather(case, chunk):
    shape, dt, sm, ss, dm, ds = case
    p = plan_of(shape, dt, sm, ss, dm, ds, chunk_bytes=chunk)
    assert B.reshard_plan_unaligned_gather_chunks(p) > 0, "case should take the unaligned row gather"
    assert B.reshard_plan_gather_chunks(p) == 0 and B.reshard_plan_realign_chunks(p) == 0
    host_case(shape, dt, sm, ss, dm, ds, chunk_bytes=chunk)
    q = plan_of(shape, dt, sm, ss, dm, ds, flags=B.RESHARD_NO_GATHER)
    assert B.reshard_plan_unaligned_gather_chunks(q) == 0
    host_case(shape, dt, sm, ss, dm, ds, flags=B.RESHARD_NO_GATHER)


def test_unaligned_gather_declines():
    # destination rows that are not contiguous, or one sender per row with
    # both sides in the same 16-byte phase: per-task chunks instead
    for case in (((6, 10, 300), "float16", (2, 3), "RS^0S^1", (2,), "RRS^0"),
                 ((8, 64, 1024), "float16", (1,), "RRR", (4,), "RRS^0")):
        p = plan_of(*case)
        assert B.reshard_plan_unaligned_gather_chunks(p) == 0
        host_case(*case)


SHORT_SEGMENT_CASES = [
    # segments under 16 bytes: at fan-out 1 units of their own width, else
    # slots of three or more pieces
    ((4, 8, 40), "float16", (8,), "RRS^0", (2,), "S^0RR"),              # 10-byte segments
    ((3, 16, 60), "uint8", (1, 8), "RRS^1", (2,), "RRR"),              # 8/7-byte segments, fan-out 2
    ((2, 12, 27), "float32", (1, 3, 3), "RRS^{12}", (1,), "RRR"),      # 12-byte segments
    ((2, 64, 12300), "float16", (4, 8), "RRS^{01}", (4, 8), "S^0RS^1"),  # a 4-byte segment at most row starts
    ((5, 40, 33), "uint8", (1, 11), "RRS^1", (3,), "S^0RR"),           # 3-byte segments
]


@pytest.mark.parametrize("case", SHORT_SEGMENT_CASES)
@pytest.mark.parametrize("chunk", [0, 64, 1000])
def test_host_unaligned_gather_short_segments(case, chunk):
    p = plan_of(*case, chunk_bytes=chunk)
    assert B.reshard_plan_unaligned_gather_chunks(p) > 0 and B.reshard_plan_realign_chunks(p) == 0
    host_case(*case, chunk_bytes=chunk)


@pytest.mark.parametrize("case", SHORT_SEGMENT_CASES)
def test_short_segments_take_units_at_fanout_one(case):
    p = plan_of(*case)
    fanout = B.reshard_plan_stats(p)["max_fanout"]
    assert (B.reshard_plan_unit_gather_chunks(p) > 0) == (fanout == 1), fanout


def test_gather_used_by_column_split_workloads():
    for wid, w in WORKLOADS.items():
        p = plan_of(w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec)
        assert (B.reshard_plan_gather_chunks(p) > 0) == (wid in (3, 5)), wid


def test_pointer_array_marshalling():
    """pointer_array: tensors (empty ones as NULL), addresses and None, built once and passed as is."""
    import torch
    full, empty = torch.zeros(8), torch.zeros(0)
    arr = B.pointer_array([full, empty, None, 4096])
    assert isinstance(arr, ctypes.Array) and len(arr) == 4
    assert list(arr) == [full.data_ptr(), None, None, 4096]
    assert B.pointer_array(arr) is arr
    assert len(B.pointer_array([])) == 1  # never a zero-length array


def test_prebuilt_pointer_arrays_drive_the_interpreter():
    """The same plan run from lists and from pre-built arrays gives the oracle's bytes both times."""
    import torch
    shape, sm, ss, dm, ds = (8, 24, 40), (2, 2), "S^0 R S^1", (2, 2), "R S^{01} R"
    x = torch.arange(int(np.prod(shape)), dtype=torch.int32).reshape(shape).numpy()
    src = [torch.from_numpy(np.ascontiguousarray(a)) for a in oracle.shard(x, sm, ss)]
    want = oracle.reshard([s.numpy() for s in src], shape, sm, ss, dm, ds)
    p = B.reshard_plan(shape, "int32", sm, ss, dm, ds)
    for prebuilt in (False, True):
        dst = [torch.full(w.shape, -1, dtype=torch.int32) for w in want]
        sp, dp = (B.pointer_array(src), B.pointer_array(dst)) if prebuilt else (src, dst)
        B.load().reshard_debug_execute_host(p.handle, B._ptrs(sp), B._ptrs(dp))
        for g, w in zip(dst, want):
            assert np.array_equal(g.numpy(), w)
