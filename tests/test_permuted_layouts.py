"""Permuted local layouts (a buffer holds its shard as numpy.transpose(box,
perm)) and the tile-transpose chunks they need.

CPU: the planner's local shapes against the oracle's; the descriptor table
run on host memory (reshard_debug_execute_host, the kernel's tile and LDS
arithmetic with every access bounds-checked) against the oracle, bit for
bit, on seeded cases that span several tiles with ragged edges, every
element size, aligned and unaligned rows, and on argument errors.  GPU: the
kernels against the oracle on the same kinds of cases and on a transposed
activations at full size, every destination element compared, and seeded
permuted cases under random launch tunings.
"""

import random

import numpy as np
import pytest

import oracle
from paper_2211_05322_amd import binding as B
from tests.test_capi_host import run_host
from tests.test_oracle_pins import fmt_spec, random_dims

_NP = {"uint8": np.uint8, "float16": np.uint16, "float32": np.uint32, "float64": np.uint64}


def perm_cases(n, seed, big=False):
    """Random tensors (rows long enough for several 128-byte tiles), meshes,
    specs and a random permutation on each side."""
    rng = random.Random(seed)
    out = []
    while len(out) < n:
        ndim = rng.randint(2, 4)
        hi = 300 if big else 140
        shape = [rng.randint(1, 6) for _ in range(ndim)]
        for d in rng.sample(range(ndim), 2):  # two long dimensions
            shape[d] = rng.randint(20, hi)
        shape = tuple(shape)
        sm = tuple(rng.randint(1, 3) for _ in range(rng.randint(1, 2)))
        dm = tuple(rng.randint(1, 3) for _ in range(rng.randint(1, 2)))
        sp, dp = list(range(ndim)), list(range(ndim))
        rng.shuffle(sp)
        rng.shuffle(dp)
        if rng.random() < 0.2:
            sp = list(range(ndim))  # one side plain
        kw = {}
        if rng.random() < 0.4:
            kw["chunk_bytes"] = rng.choice([64, 1000, 8192, 40000])
        out.append((shape, rng.choice(list(_NP)), sm, fmt_spec(random_dims(rng, ndim, len(sm))), tuple(sp),
                    dm, fmt_spec(random_dims(rng, ndim, len(dm))), tuple(dp), kw))
    return out


def _inputs(shape, dt, sm, ss, sp, dm, ds, dp, seed):
    np_dtype = _NP[dt]
    es = np.dtype(np_dtype).itemsize
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 256, size=int(np.prod(shape)) * es, dtype=np.uint8).view(np_dtype).reshape(shape)
    src = oracle.shard(x, sm, ss, sp)
    want = oracle.reshard(src, shape, sm, ss, dm, ds, src_perm=sp, dst_perm=dp)
    return src, want


def host_perm_case(shape, dt, sm, ss, sp, dm, ds, dp, seed=0, **kw):
    src, want = _inputs(shape, dt, sm, ss, sp, dm, ds, dp, seed)
    p = B.reshard_plan(shape, dt, sm, ss, dm, ds, src_perm=sp, dst_perm=dp, **kw)
    for k, w in enumerate(want):
        assert tuple(B.reshard_plan_local_shape(p, 1, k)) == w.shape
    for k, a in enumerate(src):
        assert tuple(B.reshard_plan_local_shape(p, 0, k)) == a.shape
    got = run_host(p, src, [w.shape for w in want], _NP[dt])
    for k, (g, w) in enumerate(zip(got, want)):
        assert np.array_equal(g, w), f"destination {k} differs"
    return p


@pytest.mark.parametrize("case", perm_cases(120, 77))
def test_host_permuted_against_oracle(case):
    shape, dt, sm, ss, sp, dm, ds, dp, kw = case
    host_perm_case(shape, dt, sm, ss, sp, dm, ds, dp, **kw)


@pytest.mark.parametrize("dt", list(_NP))
@pytest.mark.parametrize("shape", [(130, 70), (128, 64), (33, 517), (5, 200, 3), (2, 40, 300)])
def test_host_transpose_tiles(dt, shape):
    # the last two dimensions swapped on the destination side only: every
    # task is a tile transpose, with ragged tiles at the ends of both
    # dimensions (and whole tiles at 128 x 64)
    nd = len(shape)
    dp = tuple(range(nd - 2)) + (nd - 1, nd - 2)
    rep = "R" * nd
    p = host_perm_case(shape, dt, (2,), "S^0" + "R" * (nd - 1), None, (2,), rep, dp)
    assert B.reshard_plan_transpose_chunks(p) > 0


def test_host_transpose_unaligned_rows():
    # fp16 rows of 37 elements (74 bytes): no tile row starts on a 16-byte
    # boundary, so elements move one by one on that side
    for shape, dp in (((37, 90), (1, 0)), ((90, 37), (1, 0)), ((3, 37, 41), (2, 1, 0))):
        p = host_perm_case(shape, "float16", (1,), "R" * len(shape), None, (2,), "S^0" + "R" * (len(shape) - 1),
                           dp)
        assert B.reshard_plan_transpose_chunks(p) > 0


def test_permuted_outer_dims_need_no_transpose():
    # same innermost dimension on both sides, outer dimensions swapped: the
    # direct path with per-side strides, no tile transposes
    p = host_perm_case((6, 5, 64), "float32", (2,), "S^0RR", (1, 0, 2), (3,), "RS^0R", (0, 1, 2))
    assert B.reshard_plan_transpose_chunks(p) == 0


def test_identity_permutation_is_the_plain_plan():
    a = B.reshard_plan((8, 64, 96), "float16", (2, 2), "S^0RS^1", (2, 2), "RS^0S^1")
    b = B.reshard_plan((8, 64, 96), "float16", (2, 2), "S^0RS^1", (2, 2), "RS^0S^1", src_perm=(0, 1, 2),
                       dst_perm=(0, 1, 2))
    assert B.reshard_plan_stats(a) == B.reshard_plan_stats(b)
    assert B.reshard_plan_transpose_chunks(b) == 0


def test_permutation_errors():
    with pytest.raises(B.ReshardError) as e:
        B.reshard_plan((4, 4), "float16", (2,), "S^0R", (2,), "RS^0", dst_perm=(0, 0))
    assert e.value.status == B.RESHARD_EINVAL
    with pytest.raises(B.ReshardError) as e:
        B.reshard_plan((4, 4), "float16", (2,), "S^0R", (2,), "RS^0", src_perm=(0, 2))
    assert e.value.status == B.RESHARD_EINVAL
    with pytest.raises(B.ReshardError) as e:
        B.reshard_plan((4, 4), "float16", (2,), "S^0R", (2,), "RS^0", dst_perm=(1, 0),
                       flags=B.RESHARD_STRATEGY_SENDRECV)
    assert e.value.status == B.RESHARD_EUNSUPPORTED


# buffers above 4 GiB: a transpose piece must keep every tile within 32-bit
# offsets of its origin, cut along A or B (whichever stride makes the span
# too long) -- planning only here, the GPU tests below run them
BIG_TRANSPOSES = [((1, 70000, 70000), "uint8", None, (0, 2, 1)),
                  ((1, 40000, 60000), "float16", (0, 2, 1), None)]


@pytest.mark.parametrize("shape,dt,sp,dp", BIG_TRANSPOSES)
def test_transpose_pieces_above_4_gib_plan(shape, dt, sp, dp):
    p = B.reshard_plan(shape, dt, (1,), "RRR", (1,), "RRR", src_perm=sp, dst_perm=dp)
    assert B.reshard_plan_transpose_chunks(p) > 0
    assert B.reshard_plan_stats(p)["n_descriptors"] == B.reshard_plan_transpose_chunks(p)


def test_tile_strides_beyond_31_bits_take_the_element_path():
    # 128 destination rows of one tile would lie 34 MB apart: the planner
    # keeps such layouts off the transpose kernel (plain element pieces)
    p = B.reshard_plan((1, 200, 34000000), "uint8", (1,), "RRR", (1,), "RRR", src_perm=(0, 2, 1))
    assert B.reshard_plan_transpose_chunks(p) == 0
    st = B.reshard_plan_stats(p)
    assert st["bytes_written"] == 200 * 34000000 and st["n_descriptors"] > 0


def test_too_many_chunks_fails_cleanly():
    # 29 GB of bytes whose source and destination orders share no run and
    # whose strides keep them off the tile path: one chunk per few bytes,
    # far beyond the descriptor budget -- refused, and lowering stops there
    import time
    t = time.time()
    with pytest.raises(B.ReshardError) as e:
        B.reshard_plan((16, 8, 5298, 42608), "uint8", (2,), "RS^{0}RR", (3,), "RRRR",
                       src_perm=(0, 2, 3, 1), dst_perm=(2, 3, 1, 0))
    assert e.value.status == B.RESHARD_EUNSUPPORTED and "2^24" in str(e.value)
    assert time.time() - t < 60


# --------------------------------------------------------------------- GPU

def _gpu_run(shape, dt, sm, ss, sp, dm, ds, dp, seed=0, **kw):
    import torch
    from tests.test_gpu_parity import Guarded
    src, want = _inputs(shape, dt, sm, ss, sp, dm, ds, dp, seed)
    p = B.reshard_plan(shape, dt, sm, ss, dm, ds, src_perm=sp, dst_perm=dp, **kw)
    sb = []
    for a in src:
        g = Guarded(a.nbytes, 0xA5)
        if a.nbytes:
            g.body().copy_(torch.from_numpy(np.ascontiguousarray(a).reshape(-1).view(np.uint8).copy()))
        sb.append(g)
    db = [Guarded(w.nbytes, 0x5A) for w in want]
    B.reshard_execute(p, [g.ptr for g in sb], [g.ptr for g in db])
    torch.cuda.synchronize()
    for k, (g, w) in enumerate(zip(db, want)):
        assert g.guards_ok(), f"destination {k}: write outside the buffer"
        got = g.body().cpu().numpy().view(w.dtype).reshape(w.shape)
        if not np.array_equal(got, w):
            bad = np.argwhere(got != w)[:5]
            raise AssertionError(f"destination {k}: {int((got != w).sum())} elements differ, first at {bad.tolist()}")
    for g in sb:
        assert g.guards_ok()
    return p


@pytest.mark.gpu
@pytest.mark.parametrize("case", perm_cases(60, 78, big=True))
def test_gpu_permuted_against_oracle(case):
    shape, dt, sm, ss, sp, dm, ds, dp, kw = case
    print(f"permuted {case}", flush=True)
    _gpu_run(shape, dt, sm, ss, sp, dm, ds, dp, **kw)


@pytest.mark.gpu
@pytest.mark.parametrize("dt", list(_NP))
@pytest.mark.parametrize("shape", [(130, 70), (128, 64), (33, 517), (5, 200, 3), (2, 40, 300), (4, 300, 257)])
def test_gpu_transpose_tiles(dt, shape):
    nd = len(shape)
    dp = tuple(range(nd - 2)) + (nd - 1, nd - 2)
    print(f"transpose tiles {dt} {shape}", flush=True)
    p = _gpu_run(shape, dt, (2,), "S^0" + "R" * (nd - 1), None, (2,), "R" * nd, dp)
    assert B.reshard_plan_transpose_chunks(p) > 0


@pytest.mark.gpu
def test_gpu_transpose_unaligned_rows():
    for shape, dp in (((37, 90), (1, 0)), ((90, 37), (1, 0)), ((3, 37, 41), (2, 1, 0))):
        print(f"unaligned transpose {shape} {dp}", flush=True)
        _gpu_run(shape, "float16", (1,), "R" * len(shape), None, (2,), "S^0" + "R" * (len(shape) - 1), dp)


def _tunings(n, seed):
    rng = random.Random(seed)
    return [{k: v for k, v in (("chunk_bytes", rng.choice([0, 64, 1000, 8192, 40000])),
                               ("block_threads", rng.choice([0, 64, 128, 256, 512])),
                               ("max_wgs_per_cu", rng.choice([0, 2, 4, -1]))) if v} for _ in range(n)]


@pytest.mark.gpu
def test_gpu_permuted_soak():
    # 1,000 more permuted layouts under new seeds, each with its own chunk
    # size and then a random launch tuning, in one test
    for i, (case, tn) in enumerate(zip(perm_cases(1000, 5151, big=True), _tunings(1000, 5152))):
        shape, dt, sm, ss, sp, dm, ds, dp, kw = case
        for k in (kw, tn):
            print(f"permuted soak {i} {case} {k}", flush=True)
            _gpu_run(shape, dt, sm, ss, sp, dm, ds, dp, seed=i, **k)


@pytest.mark.gpu
@pytest.mark.parametrize("case,tuning", list(zip(perm_cases(120, 91), _tunings(120, 92))))
def test_gpu_permuted_fuzz_tunings(case, tuning):
    # seeded permuted layouts under random chunk sizes, workgroup sizes and
    # residency caps (the tile transpose, and the direct and gather chunks
    # of permuted plans, under every launch shape)
    shape, dt, sm, ss, sp, dm, ds, dp, _ = case
    print(f"permuted fuzz {case} {tuning}", flush=True)
    _gpu_run(shape, dt, sm, ss, sp, dm, ds, dp, **tuning)


@pytest.mark.gpu
@pytest.mark.parametrize("name", ["transposed2", "transposed5"])
def test_gpu_transposed_activation_full_size(name):
    # the GPT activations fp16 [8, 1024, 4096] (2,4) S^0 R S^1 -> (2,4)
    # R S^0 S^1 and fp16 [8, 2048, 12288] (4,8) R R S^{01} -> (4,8) R S^1 R
    # (4 replicas) with the destination in [batch, hidden, seq] order, in the
    # benchmark's launch configuration: every destination element compared
    # with the tensor transposed at the oracle's boxes, on the GPU
    import torch
    from paper_2211_05322_amd.workloads import make_tensor, workload_by_name
    w = workload_by_name(name)
    print(f"transposed activation {w.shape}", flush=True)
    x = make_tensor(w.shape, w.dtype, "normal", seed=0).cuda()
    n = len(w.shape)
    sc = B.reshard_plan(w.shape, w.dtype, (1,), "R" * n, w.src_mesh, w.src_spec, src_perm=None, dst_perm=w.src_perm)
    src = B.empty_shards(sc, 1)
    B.reshard_execute(sc, [x], src)
    p = B.reshard_plan(w.shape, w.dtype, w.src_mesh, w.src_spec, w.dst_mesh, w.dst_spec, src_perm=w.src_perm,
                       dst_perm=w.dst_perm)
    assert B.reshard_plan_transpose_chunks(p) > 0
    dst = B.empty_shards(p, 1)
    B.reshard_execute(p, src, dst)
    torch.cuda.synchronize()
    dims = oracle.parse_spec(w.dst_spec, n, len(w.dst_mesh))
    xb = x.view(torch.int16)
    for k, t in enumerate(dst):
        box = oracle.device_box(w.shape, w.dst_mesh, dims, k)
        ref = xb[tuple(slice(lo, hi) for lo, hi in box)].permute(*w.dst_perm)
        assert torch.equal(t.view(torch.int16), ref), f"destination {k}"


@pytest.mark.gpu
@pytest.mark.parametrize("shape,dt,sp,dp", BIG_TRANSPOSES)
def test_gpu_transpose_above_4_gib(shape, dt, sp, dp):
    # every byte of a transposed buffer above 4 GiB against torch's permute
    import torch
    print(f"transpose above 4 GiB {shape} {dt} src_perm={sp} dst_perm={dp}", flush=True)
    bits = torch.uint8 if dt == "uint8" else torch.int16
    lo, hi = (0, 256) if dt == "uint8" else (-32768, 32768)
    g = torch.Generator(device="cuda").manual_seed(5)
    x = torch.randint(lo, hi, shape, dtype=bits, device="cuda", generator=g)
    src = x.permute(*sp).contiguous() if sp else x
    p = B.reshard_plan(shape, dt, (1,), "RRR", (1,), "RRR", src_perm=sp, dst_perm=dp)
    dst = B.empty_shards(p, 1)
    assert dst[0].numel() * dst[0].element_size() > (4 << 30)
    B.reshard_execute(p, [src], dst)
    torch.cuda.synchronize()
    ref = x.permute(*dp) if dp else x
    assert torch.equal(dst[0].view(bits), ref)
