"""reshard_execute_noalloc: the execute variant that allocates nothing.

GPU: its output equals reshard_execute's, bit for bit, on calls in a row
through the C ABI -- workload 5 at full size (the largest table of the
workloads), then smaller inputs of every other kernel kind that reads the
tables (slots and units of the unaligned row gather, direct chunks, tile
transposes), then the first plan
again on the same stream with new source data (the tables it left in the
scratch are reused) -- and the oracle's on the small inputs.  CPU: a plan
whose tables exceed the scratch is refused before any HIP call.
"""

import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2211_05322_amd import binding as B
from paper_2211_05322_amd.workloads import WORKLOADS, as_numpy_bits, make_tensor, make_workload_tensor

MAX_TABLE = 4 << 20


def _say(msg):
    print(msg, flush=True)


def test_table_above_the_scratch_is_refused():
    # 64 MiB in 256-byte chunks: 262,144 descriptors of 112 bytes, far above
    # the scratch.  The fake (aligned, non-NULL) pointers are never used: the
    # size check comes before any HIP call.
    p = B.reshard_plan((64 << 20,), "uint8", (1,), "R", (2,), "S^0", chunk_bytes=256)
    assert B.reshard_plan_stats(p)["n_descriptors"] * 112 > MAX_TABLE
    fake = B.pointer_array([1 << 20]), B.pointer_array([2 << 20, 3 << 20])
    with pytest.raises(B.ReshardError) as e:
        B.reshard_execute_noalloc(p, fake[0], fake[1], stream=0)
    assert e.value.status == B.RESHARD_EUNSUPPORTED
    assert str(MAX_TABLE) in str(e.value)


def test_header_limit_matches():
    import os
    hdr = open(os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "reshard.h")).read()
    assert "#define RESHARD_NOALLOC_MAX_TABLE_BYTES (4u << 20)" in hdr


def _scatter(w, shape, x):
    rep = "R" * len(shape)
    sc = B.reshard_plan(shape, w.dtype, (1,), rep, w.src_mesh, w.src_spec)
    src = B.empty_shards(sc, 1)
    B.reshard_execute(sc, [x], src)
    return src


def _both(plan, src, stream):
    """(reshard_execute's destination buffers, reshard_execute_noalloc's)."""
    a, b = B.empty_shards(plan, 1), B.empty_shards(plan, 1)
    for t in b:
        t.view(torch.uint8).fill_(0x5A)
    B.reshard_execute(plan, src, a, stream=stream)
    B.reshard_execute_noalloc(plan, src, b, stream=stream)
    torch.cuda.synchronize()
    return a, b


def _same(a, b, what):
    assert len(a) == len(b)
    for k, (x, y) in enumerate(zip(a, b)):
        assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)), f"{what}: destination {k} differs"


@pytest.mark.gpu
def test_noalloc_equals_execute_on_calls_in_a_row():
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    w5 = WORKLOADS[5]

    # call 1: workload 5 at full size (row gather, 2.6 MiB of tables)
    _say("noalloc call 1: workload 5 full size")
    x = make_workload_tensor(w5, seed=0, device="cuda")
    src = _scatter(w5, w5.shape, x)
    big = B.reshard_plan(w5.shape, w5.dtype, w5.src_mesh, w5.src_spec, w5.dst_mesh, w5.dst_spec)
    assert B.reshard_plan_stats(big)["n_descriptors"] * 112 > (2 << 20)
    a, b = _both(big, src, stream)
    _same(a, b, "workload 5")
    del a, b

    # calls 2 to 5: smaller inputs, other kernel kinds (unaligned row gather
    # over slots and over units, direct chunks, tile transposes), also
    # checked against the oracle
    one_rep = ((1, 8), "R S^1 R")
    for shape, w, dst, perm, label in (((2, 64, 390), w5, None, None, "unaligned row gather"),
                                       ((2, 64, 390), w5, one_rep, None, "unit gather"),
                                       ((4, 8, 66, 16), WORKLOADS[4], None, None, "direct"),
                                       ((2, 64, 1024), w5, None, (0, 2, 1), "tile transpose")):
        _say(f"noalloc smaller call: {label} {shape}")
        dm, ds = dst or (w.dst_mesh, w.dst_spec)
        xs = make_tensor(shape, w.dtype, "normal", seed=1)
        xb = as_numpy_bits(xs)
        want = oracle.reshard(oracle.shard(xb, w.src_mesh, w.src_spec), shape, w.src_mesh, w.src_spec,
                              dm, ds, dst_perm=perm)
        p = B.reshard_plan(shape, w.dtype, w.src_mesh, w.src_spec, dm, ds, dst_perm=perm)
        kind = {"unit gather": B.reshard_plan_unit_gather_chunks,
                "tile transpose": B.reshard_plan_transpose_chunks}.get(label)
        assert kind is None or kind(p) > 0, label
        sd = _scatter(w, shape, xs.cuda())
        a, b = _both(p, sd, stream)
        _same(a, b, label)
        for k, (t, ref) in enumerate(zip(b, want)):
            got = as_numpy_bits(t).reshape(ref.shape)
            assert np.array_equal(got, ref), f"{label}: destination {k} differs from the oracle"

    # call 6: the first plan again on the same stream after another plan
    # took the scratch, new source data
    _say("noalloc call 6: workload 5 again, new data")
    x2 = make_workload_tensor(w5, seed=7, device="cuda")
    src2 = _scatter(w5, w5.shape, x2)
    a, b = _both(big, src2, stream)
    _same(a, b, "workload 5 again")

    # call 7: the same plan on the same stream right after (tables reused)
    _say("noalloc call 7: workload 5, tables in place")
    b2 = B.empty_shards(big, 1)
    B.reshard_execute_noalloc(big, src2, b2, stream=stream)
    torch.cuda.synchronize()
    _same(a, b2, "workload 5, tables reused")


@pytest.mark.gpu
def test_noalloc_on_two_streams_in_turn():
    # the same plan on another stream copies its tables on that stream first
    torch.cuda.set_device(0)
    w = WORKLOADS[5]
    shape = (2, 64, 1024)
    xs = make_tensor(shape, w.dtype, "normal", seed=3)
    p = B.reshard_plan(shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec)
    sd = _scatter(w, shape, xs.cuda())
    torch.cuda.synchronize()
    ref, _ = _both(p, sd, torch.cuda.current_stream())
    s2 = torch.cuda.Stream()
    for stream in (s2, torch.cuda.current_stream(), s2):
        out = B.empty_shards(p, 1)
        with torch.cuda.stream(stream):
            B.reshard_execute_noalloc(p, sd, out, stream=stream)
        torch.cuda.synchronize()
        _same(ref, out, "second stream")
