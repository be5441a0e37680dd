"""GPU parity: the HIP kernel (through the C ABI) against the CPU oracle.

Bit-exact comparison (raw bits) of every destination buffer.  Device
buffers sit inside larger allocations with guard bands that must stay
untouched.  Full-size workloads run in the launch configuration bench.py
times (default plan options).
"""

import os
import random
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_2211_05322_amd import binding as B
from paper_2211_05322_amd.workloads import (UNEVEN_WORKLOADS, WORKLOADS, as_numpy_bits, make_workload_tensor,
                                            workload_by_name)
from tests.test_capi_host import _fuzz, _fuzz_lowering
from tests.test_oracle_pins import fmt_spec, random_dims

pytestmark = pytest.mark.gpu

GUARD = 256  # bytes on each side of every device buffer
_T = {"uint8": torch.uint8, "float16": torch.float16, "float32": torch.float32, "float64": torch.float64,
      "bfloat16": torch.bfloat16, "int16": torch.int16, "int32": torch.int32, "int64": torch.int64}


def _say(msg):
    print(msg, flush=True)


class Guarded:
    """A device buffer of `nbytes` inside an allocation with guard bands."""

    def __init__(self, nbytes, fill):
        self.nbytes = nbytes
        self.raw = torch.full((nbytes + 2 * GUARD,), fill, dtype=torch.uint8, device="cuda")
        self.fill = fill

    @property
    def ptr(self):
        return self.raw.data_ptr() + GUARD if self.nbytes else None

    def body(self):
        return self.raw[GUARD:GUARD + self.nbytes]

    def guards_ok(self):
        return bool((self.raw[:GUARD] == self.fill).all()) and bool((self.raw[GUARD + self.nbytes:] == self.fill).all())


def run_gpu(shape, dtype, sm, ss, dm, ds, x_cpu, flags=0, stream=None, **kw):
    """Shard x on the host (oracle), run the kernel, return (got, want) raw-bit arrays."""
    x = as_numpy_bits(x_cpu)
    es = x.dtype.itemsize
    src = oracle.shard(x, sm, ss)
    want = oracle.reshard(src, shape, sm, ss, dm, ds)
    p = B.reshard_plan(shape, dtype, sm, ss, dm, ds, flags=flags, **kw)
    sbufs = []
    for a in src:
        g = Guarded(a.nbytes, 0xA5)
        if a.nbytes:
            g.body().copy_(torch.from_numpy(a.reshape(-1).view(np.uint8).copy()))
        sbufs.append(g)
    dbufs = [Guarded(w.nbytes, 0x5A) for w in want]
    B.reshard_execute(p, [g.ptr for g in sbufs], [g.ptr for g in dbufs], stream=stream)
    torch.cuda.synchronize()
    got = []
    for g, w in zip(dbufs, want):
        assert g.guards_ok(), "kernel wrote outside a destination buffer"
        got.append(g.body().cpu().numpy().view(f"u{es}").reshape(w.shape))
    for g, a in zip(sbufs, src):
        assert g.guards_ok()
        if a.nbytes:
            assert np.array_equal(g.body().cpu().numpy(), a.reshape(-1).view(np.uint8)), "source modified"
    return got, want


def assert_same(got, want):
    assert len(got) == len(want)
    for k, (g, w) in enumerate(zip(got, want)):
        assert g.shape == w.shape, k
        if not np.array_equal(g, w):
            bad = np.argwhere(g != w)[:5]
            raise AssertionError(f"buffer {k}: {int((g != w).sum())} elements differ, first at {bad.tolist()}")


def rand_bits(shape, dtype, seed):
    g = torch.Generator().manual_seed(seed)
    es = torch.empty((), dtype=_T[dtype]).element_size()
    n = int(np.prod(shape)) if shape else 1
    raw = torch.randint(0, 256, (n * es,), generator=g, dtype=torch.uint8)
    return raw.view(_T[dtype]).reshape(shape)


def test_single_hip_runtime_in_process():
    B.load()
    torch.zeros(1, device="cuda")
    maps = open("/proc/self/maps").read()
    paths = {line.split()[-1] for line in maps.splitlines() if "libamdhip64" in line}
    assert len(paths) == 1, paths


def test_fig2_on_gpu():
    _say("fig2")
    x = torch.arange(16, dtype=torch.float32).reshape(4, 4)
    got, want = run_gpu((4, 4), "float32", (2, 2), "S^{01}R", (2, 2), "S^0R", x)
    assert_same(got, want)


@pytest.mark.parametrize("case", range(1, 10))
def test_table3_scaled(case):
    import json
    here = os.path.dirname(__file__)
    c = json.load(open(os.path.join(here, "golden", "table3_cases.json")))["cases"][case - 1]
    shape = (64, 48, 40)
    _say(f"table3 case {case} {shape}")
    for flags in (0, B.RESHARD_SENDER_NAIVE):
        x = rand_bits(shape, "float16", case)
        got, want = run_gpu(shape, "float16", tuple(c["send_mesh"]), c["send_spec"], tuple(c["recv_mesh"]),
                            c["recv_spec"], x, flags=flags)
        assert_same(got, want)


@pytest.mark.parametrize("case", _fuzz(60, 5))
def test_fuzz_small(case):
    shape, dt, sm, ss, dm, ds, flags = case
    _say(f"fuzz {case}")
    got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, 3), flags=flags)
    assert_same(got, want)


def _mid_cases(n, seed):
    rng = random.Random(seed)
    out = []
    while len(out) < n:
        ndim = rng.randint(2, 4)
        shape = tuple(rng.choice([1, 3, 17, 64, 97, 130, 256]) for _ in range(ndim))
        if int(np.prod(shape)) > 3_000_000:
            continue
        sm = tuple(rng.randint(1, 4) for _ in range(2))
        dm = tuple(rng.randint(1, 4) for _ in range(2))
        out.append((shape, rng.choice(["uint8", "float16", "float32", "float64"]), sm,
                    fmt_spec(random_dims(rng, ndim, 2)), dm, fmt_spec(random_dims(rng, ndim, 2))))
    return out


@pytest.mark.parametrize("case", _mid_cases(24, 77))
def test_fuzz_multi_tile_ragged(case):
    # sizes spanning many chunks with ragged tails and misaligned phases
    shape, dt, sm, ss, dm, ds = case
    _say(f"mid {case}")
    for kw in ({}, {"chunk_bytes": 1000, "block_threads": 64, "max_wgs_per_cu": 2},
               {"chunk_bytes": 70000, "block_threads": 1024, "max_wgs_per_cu": -1}):
        got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, 4), **kw)
        assert_same(got, want)


@pytest.mark.parametrize("flags", [B.RESHARD_XCD_REMAP, B.RESHARD_TASK_ORDER,
                                   B.RESHARD_XCD_REMAP | B.RESHARD_TASK_ORDER | B.RESHARD_SENDER_NAIVE])
@pytest.mark.parametrize("cap", [-1, 2, 32])
def test_launch_order_flags_and_residency_caps(flags, cap):
    w = WORKLOADS[5]
    shape = (2, 64, 384)
    x = rand_bits(shape, w.dtype, 9)
    got, want = run_gpu(shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec, x,
                        flags=flags, chunk_bytes=4096, max_wgs_per_cu=cap)
    assert_same(got, want)


def test_replicated_sources_may_share_one_buffer():
    """Sources are only read: the eight replicas of a replicated source may
    all be the same device buffer (Table 3 case 2's specs, scaled)."""
    shape, sm, ss, dm, ds = (64, 48, 40), (2, 4), "RRR", (2, 4), "S^0RR"
    x = rand_bits(shape, "float16", 5)
    xb = as_numpy_bits(x)
    want = oracle.reshard([xb] * 8, shape, sm, ss, dm, ds)
    p = B.reshard_plan(shape, "float16", sm, ss, dm, ds)
    one = x.cuda()
    dst = B.empty_shards(p, 1)
    B.reshard_execute(p, [one] * 8, dst)
    torch.cuda.synchronize()
    assert torch.equal(one.cpu().view(torch.int16), x.view(torch.int16))
    assert_same([d.cpu().numpy().view(np.uint16) for d in dst], want)


def test_special_bit_patterns():
    bits = np.array([0x7E01, 0xFE02, 0x8000, 0x7C00, 0xFC00, 0x0001, 0x7FFF, 0xFFFF] * 64, dtype=np.uint16)
    x = torch.from_numpy(bits.view(np.float16).reshape(16, 32).copy())
    got, want = run_gpu((16, 32), "float16", (2,), "S^0R", (2, 2), "RS^1", x)
    assert_same(got, want)


def test_empty_shards_null_pointers_and_empty_tensor():
    x = rand_bits((3, 40), "float32", 1)
    got, want = run_gpu((3, 40), "float32", (4,), "S^0R", (2,), "RS^0", x)
    assert_same(got, want)
    p = B.reshard_plan((0, 4), "float32", (2,), "S^0R", (2,), "RS^0")
    B.reshard_execute(p, [None, None], [None, None])
    torch.cuda.synchronize()


def test_misaligned_pointer_rejected():
    p = B.reshard_plan((8, 64), "float16", (2,), "S^0R", (2,), "RS^0")
    assert B.reshard_plan_alignment(p) == 16
    a = torch.zeros(1024, dtype=torch.uint8, device="cuda")
    src = [a.data_ptr() + 2, a.data_ptr() + 512]
    with pytest.raises(B.ReshardError) as e:
        B.reshard_execute(p, src, [a.data_ptr(), a.data_ptr() + 512])
    assert e.value.status == B.RESHARD_EINVAL


def test_plan_reuse_on_streams():
    shape = (64, 256)
    x = rand_bits(shape, "float32", 2)
    xs = as_numpy_bits(x)
    src = oracle.shard(xs, (2, 2), "S^0S^1")
    want = oracle.reshard(src, shape, (2, 2), "S^0S^1", (4,), "RS^0")
    p = B.reshard_plan(shape, "float32", (2, 2), "S^0S^1", (4,), "RS^0")
    sd = [torch.from_numpy(a.copy()).cuda() for a in src]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for s in (s1, s2, None, s1):
        dd = [torch.empty(w.shape, dtype=torch.int32, device="cuda") for w in want]
        B.reshard_execute(p, sd, dd, stream=s)
        torch.cuda.synchronize()
        for d, w in zip(dd, want):
            assert np.array_equal(d.cpu().numpy().view(np.uint32), w)


@pytest.mark.parametrize("wid", sorted(WORKLOADS) + sorted(UNEVEN_WORKLOADS))
def test_workload_full_size(wid):
    """Full-size workload, bench launch configuration, every output compared."""
    w = workload_by_name(wid)
    _say(f"workload {wid} {w.name} {w.shape}")
    x = make_workload_tensor(w, seed=0)
    xb = as_numpy_bits(x)
    es = xb.dtype.itemsize
    src = oracle.shard(xb, w.src_mesh, w.src_spec)
    del xb
    want = oracle.reshard(src, w.shape, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec)
    p = B.reshard_plan(w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec)
    sd = [torch.from_numpy(a).cuda() for a in src]
    del src
    dd = B.empty_shards(p, 1)
    for d in dd:
        d.view(torch.uint8 if es == 1 else torch.int16 if es == 2 else torch.int32).fill_(-1 if es > 1 else 255)
    B.reshard_execute(p, sd, dd)
    torch.cuda.synchronize()
    for k, (d, wnt) in enumerate(zip(dd, want)):
        g = as_numpy_bits(d)
        assert g.shape == wnt.shape
        assert np.array_equal(g, wnt), f"workload {wid} destination {k} differs"
    _say(f"workload {wid} ok")


# ------------------------------------------------------ LDS realignment path

from tests.test_capi_host import REALIGN_CASES  # noqa: E402


@pytest.mark.parametrize("case", REALIGN_CASES)
def test_realign_path(case):
    shape, dt, sm, ss, dm, ds = case
    _say(f"realign {case}")
    ng = B.RESHARD_NO_GATHER  # some cases take the unaligned row gather by default
    assert B.reshard_plan_realign_chunks(B.reshard_plan(shape, dt, sm, ss, dm, ds, flags=ng)) > 0
    for kw in ({}, {"flags": ng}, {"chunk_bytes": 100, "block_threads": 64, "flags": ng},
               {"chunk_bytes": 5000, "block_threads": 1024, "flags": ng},
               {"max_wgs_per_cu": -1, "flags": ng}, {"flags": B.RESHARD_TASK_ORDER | B.RESHARD_XCD_REMAP | ng},
               {"flags": B.RESHARD_NO_REALIGN | ng}, {"flags": B.RESHARD_LDS_STAGING | ng},
               {"flags": B.RESHARD_LDS_STAGING | ng, "chunk_bytes": 300, "block_threads": 64}):
        got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, 5), **kw)
        assert_same(got, want)


def test_realign_uneven_large():
    # fp16 [4, 512, 12300] over 32 shards of the last dim (385 or 384 wide):
    # every row phase differs between the two layouts; by default the
    # unaligned row gather, else mixed direct and realignment chunks
    shape = (4, 512, 12300)
    sm, ss, dm, ds = (4, 8), "RRS^{01}", (4, 8), "RS^1R"
    _say("realign uneven large")
    p = B.reshard_plan(shape, "float16", sm, ss, dm, ds, flags=B.RESHARD_NO_GATHER)
    assert B.reshard_plan_realign_chunks(p) > 0
    assert B.reshard_plan_unaligned_gather_chunks(B.reshard_plan(shape, "float16", sm, ss, dm, ds)) > 0
    for flags in (0, B.RESHARD_NO_GATHER, B.RESHARD_NO_GATHER | B.RESHARD_LDS_STAGING):
        got, want = run_gpu(shape, "float16", sm, ss, dm, ds, rand_bits(shape, "float16", 6), flags=flags)
        assert_same(got, want)


# ------------------------------------------ comparison strategies (f2)

@pytest.mark.parametrize("strategy", [B.RESHARD_STRATEGY_SENDRECV, B.RESHARD_STRATEGY_ALLGATHER])
@pytest.mark.parametrize("case", _mid_cases(8, 91))
def test_strategies(strategy, case):
    shape, dt, sm, ss, dm, ds = case
    _say(f"strategy {strategy} {case}")
    got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, 8), flags=strategy)
    assert_same(got, want)


@pytest.mark.parametrize("strategy", [B.RESHARD_STRATEGY_SENDRECV, B.RESHARD_STRATEGY_ALLGATHER])
def test_strategies_full_size_fanout8(strategy):
    w = WORKLOADS[3]  # 8 receivers per slice
    _say(f"strategy {strategy} workload 3")
    x = make_workload_tensor(w, seed=1)
    xb = as_numpy_bits(x)
    src = oracle.shard(xb, w.src_mesh, w.src_spec)
    want = oracle.reshard(src, w.shape, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec)
    p = B.reshard_plan(w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec, flags=strategy)
    sd = [torch.from_numpy(a).cuda() for a in src]
    dd = B.empty_shards(p, 1)
    B.reshard_execute(p, sd, dd)
    torch.cuda.synchronize()
    for k, (d, wnt) in enumerate(zip(dd, want)):
        assert np.array_equal(as_numpy_bits(d), wnt), f"destination {k}"


# ------------------------------------------------------------ row gather

from tests.test_capi_host import GATHER_CASES  # noqa: E402


@pytest.mark.parametrize("case", GATHER_CASES)
def test_gather_path(case):
    shape, dt, sm, ss, dm, ds = case
    _say(f"gather {case}")
    assert B.reshard_plan_gather_chunks(B.reshard_plan(shape, dt, sm, ss, dm, ds)) > 0
    for kw in ({}, {"chunk_bytes": 256, "block_threads": 64}, {"chunk_bytes": 3000, "block_threads": 1024},
               {"max_wgs_per_cu": -1}, {"flags": B.RESHARD_XCD_REMAP}, {"flags": B.RESHARD_NO_GATHER},
               {"gather_band": 1}, {"gather_band": 3, "chunk_bytes": 1024}):
        got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, 12), **kw)
        assert_same(got, want)


# ------------------------------------------------- unaligned row gather

from tests.test_capi_host import SHORT_SEGMENT_CASES, UNALIGNED_GATHER_CASES  # noqa: E402


@pytest.mark.parametrize("case", SHORT_SEGMENT_CASES + [((4, 41, 77), "float16", (2, 2), "R S^0 S^1", (2,), "S^0 R R")])
def test_unaligned_gather_short_segments_and_runs(case):
    # segments under 16 bytes (at fan-out 1 units of their own width, else
    # slots of three or more pieces) and runs shorter than a chunk, on the
    # unaligned row gather
    shape, dt, sm, ss, dm, ds = case
    _say(f"short segments / runs {case}")
    assert B.reshard_plan_unaligned_gather_chunks(B.reshard_plan(shape, dt, sm, ss, dm, ds)) > 0
    for kw in ({}, {"chunk_bytes": 64, "block_threads": 64}, {"chunk_bytes": 1000}, {"max_wgs_per_cu": -1}):
        got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, 15), **kw)
        assert_same(got, want)


@pytest.mark.parametrize("case", UNALIGNED_GATHER_CASES)
def test_unaligned_gather_path(case):
    shape, dt, sm, ss, dm, ds = case
    _say(f"unaligned gather {case}")
    assert B.reshard_plan_unaligned_gather_chunks(B.reshard_plan(shape, dt, sm, ss, dm, ds)) > 0
    for kw in ({}, {"chunk_bytes": 64, "block_threads": 64}, {"chunk_bytes": 3000, "block_threads": 1024},
               {"max_wgs_per_cu": -1}, {"max_wgs_per_cu": 2}, {"flags": B.RESHARD_XCD_REMAP},
               {"flags": B.RESHARD_NO_GATHER}):
        got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, 14), **kw)
        assert_same(got, want)


@pytest.mark.parametrize("shape,n,dm", [
    # fan-out 2 (destination slots, 64 per 1 KiB chunk)
    ((2, 83, 390), 127, (2,)), ((8, 21, 390), 128, (2,)), ((13, 13, 390), 129, (2,)),
    ((2, 167, 390), 255, (2,)), ((1, 337, 390), 257, (2,)),
    # fan-out 1 (unit gather: 32 segments of 2 units a row, one row per 1 KiB chunk)
    ((1, 127, 390), 127, (1,)), ((2, 64, 390), 128, (1,)), ((1, 129, 390), 129, (1,)),
    ((5, 51, 390), 255, (1,)), ((1, 257, 390), 257, (1,))])
def test_unaligned_gather_chunk_counts_around_xcd_runs(shape, n, dm):
    """The unaligned row gather hands chunks to the XCDs in runs of 16, on a
    grid rounded up to whole rounds of 8 x 16 chunks: counts just below, at
    and above such a round, with and without the XCD flag, one row group
    gathered from 32 senders (26/24-byte segments)."""
    args = (shape, "float16", (4, 8), "R R S^{01}", dm, "R R R")
    _say(f"unaligned gather, {n} chunks: {shape} -> {dm}")
    assert B.reshard_plan_unaligned_gather_chunks(B.reshard_plan(*args, chunk_bytes=1024)) == n
    for flags in (0, B.RESHARD_XCD_REMAP):
        got, want = run_gpu(*args, rand_bits(shape, "float16", n), flags=flags, chunk_bytes=1024)
        assert_same(got, want)


from tests.test_capi_host import RUN_CASES  # noqa: E402


@pytest.mark.parametrize("case", RUN_CASES)
def test_unaligned_gather_in_runs(case):
    """Destination rows contiguous only in runs: one region per run."""
    shape, dt, sm, ss, dm, ds = case
    _say(f"unaligned gather in runs {case}")
    for kw in ({}, {"chunk_bytes": 256}, {"chunk_bytes": 1024, "block_threads": 64}, {"chunk_bytes": 1024},
               {"chunk_bytes": 1024, "flags": B.RESHARD_XCD_REMAP}):
        got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, 23), **kw)
        assert_same(got, want)


@pytest.mark.parametrize("dm", [(2,), (2, 2), (2, 4)])
def test_unaligned_gather_in_runs_larger(dm):
    """fp16 [4, 511, 1029]: 2058-byte rows, the middle dimension split 256/255
    on the source and the outer one on the destination -- runs of 256 or 255
    rows in different 16-byte phases, fan-out 1, 2 and 4."""
    shape, sm, ss, ds = (4, 511, 1029), (2,), "R S^0 R", "S^0 R R"
    _say(f"unaligned gather in runs {shape} -> {dm}")
    p = B.reshard_plan(shape, "float16", sm, ss, dm, ds)
    assert B.reshard_plan_unaligned_gather_chunks(p) > 0 and B.reshard_plan_realign_chunks(p) == 0
    got, want = run_gpu(shape, "float16", sm, ss, dm, ds, rand_bits(shape, "float16", 29))
    assert_same(got, want)


# ------------------------------------------------------------ maximum sizes

def test_max_buffers_direct_and_gather():
    """496 buffers (the compiled limit): the large kernel-argument block, on
    the direct path (fan-out 2) and on the row-gather path (248 senders per
    destination row)."""
    for case in (((496, 248), "float32", (248,), "S^0R", (2, 124), "RS^1"),
                 ((248, 992), "float32", (248,), "RS^0", (2, 124), "S^1R")):
        shape, dt, sm, ss, dm, ds = case
        _say(f"max buffers {case}")
        p = B.reshard_plan(shape, dt, sm, ss, dm, ds)
        assert p.n_src + p.n_dst == 496
        if ss == "RS^0":
            assert B.reshard_plan_gather_chunks(p) > 0
        got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, 21))
        assert_same(got, want)


def _check_against_boxes(x, dst, shape, mesh, spec):
    """Destination k must equal x sliced at the oracle's box of device k."""
    dims = oracle.parse_spec(spec, len(shape), len(mesh))
    for k, d in enumerate(dst):
        box = oracle.device_box(shape, mesh, dims, k)
        want = x[tuple(slice(lo, hi) for lo, hi in box)]
        assert tuple(d.shape) == tuple(want.shape)
        assert torch.equal(d.view(torch.int16), want.view(torch.int16)), f"destination {k} differs"


def _table3():
    import json
    return json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "table3_cases.json")))


@pytest.mark.parametrize("case", range(1, 10))
def test_table3_full_size_on_gpu(case):
    """Table 3's nine cases at the tensor size Section 5.1.2 gives,
    (1024, 1024, 512) (fp16, the element type the paper leaves open; 1 GiB),
    with the readings of its garbled entries: each source shard is the tensor
    sliced at the oracle's box, and every destination element is compared on
    the GPU with the tensor sliced at the oracle's destination box."""
    g = _table3()
    c = g["cases"][case - 1]
    shape = tuple(g["tensor_shape"])
    sm, ss, dm, ds = tuple(c["send_mesh"]), c["send_spec"], tuple(c["recv_mesh"]), c["recv_spec"]
    _say(f"table 3 case {case} at {shape}: {sm} {ss} -> {dm} {ds}")
    x = make_workload_tensor(WORKLOADS[5].__class__("t3", shape, "float16", "bits", sm, ss, dm, ds),
                             seed=case, device="cuda")
    dims = oracle.parse_spec(ss, len(shape), len(sm))
    src = []
    for k in range(int(np.prod(sm))):
        box = oracle.device_box(shape, sm, dims, k)
        src.append(x[tuple(slice(lo, hi) for lo, hi in box)].contiguous())
    p = B.reshard_plan(shape, "float16", sm, ss, dm, ds)
    dst = B.empty_shards(p, 1)
    for d in dst:
        d.view(torch.int16).fill_(-1)
    B.reshard_execute(p, src, dst)
    torch.cuda.synchronize()
    del src
    _check_against_boxes(x, dst, shape, dm, ds)
    del x, dst
    torch.cuda.empty_cache()


@pytest.mark.parametrize("case", [
    # one 5 GiB source to two 5 GiB replicas (offsets past 2^32 on both sides)
    ((5, 1 << 29), (1,), "RR", (2,), "RR"),
    # two senders' 512 MiB column halves gathered into 1 GiB rows of one 5 GiB buffer
    ((5, 1 << 29), (2,), "RS^0", (1,), "RR"),
    # rows of 2^30 + 10 bytes split unevenly: different 16-byte phases, 5 GiB source
    ((5, (1 << 29) + 5), (1,), "RR", (2,), "RS^0"),
    # the same rows gathered from two uneven, misaligned column halves into one 5 GiB buffer
    ((5, (1 << 29) + 5), (2,), "RS^0", (1,), "RR"),
])
def test_over_4gib(case):
    """Buffers above 4 GiB: every destination compared, element by element on
    the GPU, with the tensor sliced at the oracle's shard boxes."""
    shape, sm, ss, dm, ds = case
    _say(f"over 4 GiB {case}")
    x = make_workload_tensor(WORKLOADS[5].__class__("big", shape, "float16", "bits", sm, ss, dm, ds),
                             seed=3, device="cuda")
    dims = oracle.parse_spec(ss, len(shape), len(sm))
    src = []
    for k in range(int(np.prod(sm))):
        box = oracle.device_box(shape, sm, dims, k)
        src.append(x[tuple(slice(lo, hi) for lo, hi in box)].contiguous())
    p = B.reshard_plan(shape, "float16", sm, ss, dm, ds)
    dst = B.empty_shards(p, 1)
    for d in dst:
        d.view(torch.int16).fill_(-1)
    B.reshard_execute(p, src, dst)
    torch.cuda.synchronize()
    del src
    _check_against_boxes(x, dst, shape, dm, ds)
    _say(f"over 4 GiB {case} ok")
    del x, dst
    torch.cuda.empty_cache()


# ------------------------------------------------------------- HIP graphs

@pytest.mark.parametrize("case", [
    ((2, 64, 1024), "float16", (4, 8), "RRS^{01}", (4, 8), "RS^1R"),      # row gather
    ((2, 64, 12300), "float16", (4, 8), "RRS^{01}", (4, 8), "RS^1R"),     # unaligned row gather
    ((4, 96, 70), "float16", (2,), "S^0RR", (2, 2), "RS^0S^1"),           # realignment
    ((8, 1024, 64), "float32", (2, 4), "S^0RS^1", (2, 4), "RS^0S^1"),     # direct
])
def test_graph_capture_and_replay(case):
    """An execute captured into a HIP graph (after reshard_plan_upload) replays
    correctly: new source data between replays, eager work on the stream in
    between, every replay checked."""
    shape, dt, sm, ss, dm, ds = case
    _say(f"graph {case}")
    p = B.reshard_plan(shape, dt, sm, ss, dm, ds)
    es = np.dtype({"float16": np.uint16, "float32": np.uint32}[dt]).itemsize
    ui = {2: torch.int16, 4: torch.int32}[es]
    src = B.empty_shards(p, 0)
    dst = B.empty_shards(p, 1)
    B.reshard_plan_upload(p)  # the table upload happens outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        B.reshard_execute(p, src, dst)
    scratch = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    for rep in range(4):
        x = rand_bits(shape, dt, 40 + rep)
        xs = oracle.shard(as_numpy_bits(x), sm, ss)
        want = oracle.reshard(xs, shape, sm, ss, dm, ds)
        for buf, a in zip(src, xs):
            if a.size:
                buf.copy_(torch.from_numpy(a.view(f"i{es}").copy()).view(buf.dtype).reshape(buf.shape))
        for d in dst:
            d.view(ui).fill_(-1)
        scratch.fill_(rep)  # eager work between replays
        g.replay()
        torch.cuda.synchronize()
        for k, (d, w) in enumerate(zip(dst, want)):
            assert np.array_equal(as_numpy_bits(d), w), f"replay {rep} destination {k}"
    del g


# ----------------------------------------------------- concurrent callers

def test_concurrent_executes_share_one_plan():
    """Four host threads call reshard_execute on one fresh plan at once, each
    on its own stream and destination buffers: the table upload happens once
    (under the plan's lock) and every output is bit-exact."""
    import threading

    shape, dt, sm, ss, dm, ds = (4, 64, 1024), "float16", (4, 8), "RRS^{01}", (4, 8), "RS^1R"
    _say("concurrent executes")
    x = rand_bits(shape, dt, 77)
    xs = oracle.shard(as_numpy_bits(x), sm, ss)
    want = oracle.reshard(xs, shape, sm, ss, dm, ds)
    p = B.reshard_plan(shape, dt, sm, ss, dm, ds)
    src = [torch.from_numpy(a.view("i2").copy()).cuda() for a in xs]
    outs = [[torch.full(w.shape, -1, dtype=torch.int16, device="cuda") for w in want] for _ in range(4)]
    streams = [torch.cuda.Stream() for _ in range(4)]
    torch.cuda.synchronize()
    errors = []
    start = threading.Barrier(4)

    def worker(i):
        try:
            start.wait()
            for _ in range(3):
                B.reshard_execute(p, src, outs[i], stream=streams[i])
        except Exception as e:  # reported below
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for i in range(4):
        for k, (d, w) in enumerate(zip(outs[i], want)):
            assert np.array_equal(d.cpu().numpy().view(np.uint16), w), f"thread {i} destination {k}"


# ------------------------------------------- lowering flags x tunings fuzz

@pytest.mark.parametrize("case", _fuzz_lowering(400, 2024))
def test_fuzz_lowering_flags_and_tunings(case):
    shape, dt, sm, ss, dm, ds, kw = case
    _say(f"lowering fuzz {case}")
    got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, zlib.crc32(repr(case).encode())), **kw)
    assert_same(got, want)


def test_fuzz_lowering_soak():
    # 3,000 more cases of the generator above under a second seed, in one
    # test (each printed before it runs)
    for i, case in enumerate(_fuzz_lowering(3000, 90210)):
        shape, dt, sm, ss, dm, ds, kw = case
        _say(f"lowering soak {i} {case}")
        got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, zlib.crc32(repr(case).encode())), **kw)
        assert_same(got, want)


@pytest.mark.parametrize("dt", ["bfloat16", "int16", "int32", "int64"])
def test_other_element_types(dt):
    """The kernels see only the element size: bf16 and the integer types go
    through the same paths bit for bit (row gather and realignment cases)."""
    for shape, sm, ss, dm, ds in (((2, 16, 512), (4, 8), "RRS^{01}", (4, 8), "RS^1R"),
                                  ((3, 40, 333), (2, 2), "RS^0S^1", (3,), "RRS^0")):
        _say(f"dtype {dt} {shape}")
        got, want = run_gpu(shape, dt, sm, ss, dm, ds, rand_bits(shape, dt, 31))
        assert_same(got, want)
