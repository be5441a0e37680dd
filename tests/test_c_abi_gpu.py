"""The C ABI on the GPU from a C program: `tests/c/abi_gpu.c` (built by
`paper_2211_05322_amd.build.build_c_client`) plans and executes through
include/reshard.h with device memory and streams from the HIP runtime
itself, in a process without Python or torch.  Its destination bytes are
compared bit for bit with the oracle; the client itself checks guard bands
and that the sources are unmodified.

The cases cover each kernel kind (direct, aligned and unaligned row gather,
realignment), 1024-thread workgroups (whose residency reservation raises
the kernel's LDS limit), the null stream and a created one, an explicit
upload before executing, repeated executes, empty shards passed as NULL and
more than 64 buffers (the 496-pointer argument block)."""

import os
import subprocess
import zlib

import numpy as np
import pytest

import oracle
from paper_2211_05322_amd import build as _build

pytestmark = pytest.mark.gpu

# reshard_dtype_t codes of include/reshard.h; flags 0x100 = RESHARD_NO_GATHER,
# 0x10 = RESHARD_LDS_STAGING
_CODE = {"uint8": 0, "float16": 2, "float32": 4, "int64": 7}

# (name, shape, dtype, src mesh, src spec, dst mesh, dst spec, block, stream, upload, repeat, flags)
CASES = [
    ("direct_fp32_mesh1x2_to_2x2", (256, 1024), "float32", (1, 2), "S^1 R", (2, 2), "R S^0", 0, 0, 0, 1, 0),
    ("row_gather_fp16_4x8_to_4x8", (2, 64, 1024), "float16", (4, 8), "R R S^{01}", (4, 8), "R S^1 R",
     0, 1, 1, 2, 0),
    ("unaligned_gather_fp16_4x8_to_4x8", (2, 64, 390), "float16", (4, 8), "R R S^{01}", (4, 8), "R S^1 R",
     0, 1, 0, 1, 0),
    ("unaligned_gather_single_sender_u8", (4, 130, 101), "uint8", (2, 4), "S^0 R S^1", (2, 4), "R S^0 S^1",
     0, 0, 0, 1, 0),
    ("direct_block1024_uneven_h", (8, 64, 66, 64), "float16", (2, 2), "S^0 S^1 R R", (4, 2), "R R S^0 R",
     1024, 1, 0, 1, 0),
    ("realign_shifted_loads_u8", (4, 130, 101), "uint8", (2,), "R S^0 R", (2,), "S^0 R R", 0, 0, 0, 1, 0x100),
    ("realign_lds_staging_u8", (4, 130, 101), "uint8", (2,), "R S^0 R", (2,), "S^0 R R", 0, 1, 0, 1, 0x110),
    ("unaligned_gather_in_runs_u8", (4, 130, 101), "uint8", (2,), "R S^0 R", (2,), "S^0 R R", 0, 0, 0, 1, 0),
    ("empty_shards_int64", (3, 40), "int64", (4,), "S^0 R", (2, 2), "R S^1", 0, 0, 0, 1, 0),
    ("many_buffers_16x16_to_8x8", (32, 64), "float16", (16, 16), "S^0 S^1", (8, 8), "S^1 R", 0, 1, 1, 1, 0),
]


def _spec_token(spec):
    return ",".join(spec.split())


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_c_client_matches_oracle(case, tmp_path, gpu_lib):
    name, shape, dt, sm, ss, dm, ds, block, stream, upload, repeat, flags = case
    exe = _build.C_CLIENT
    assert os.path.exists(exe), f"{exe} missing: run paper_2211_05322_amd.build (or __graft_entry__.build())"
    es = np.dtype(dt).itemsize
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    x = rng.integers(0, 256, size=int(np.prod(shape)) * es, dtype=np.uint8).view(dt).reshape(shape)
    src = oracle.shard(x, sm, ss)
    want = oracle.reshard(src, shape, sm, ss, dm, ds)
    (tmp_path / "case.txt").write_text(
        f"dtype {_CODE[dt]}\nshape {len(shape)} {' '.join(map(str, shape))}\n"
        f"src {len(sm)} {' '.join(map(str, sm))} {_spec_token(ss)}\n"
        f"dst {len(dm)} {' '.join(map(str, dm))} {_spec_token(ds)}\n"
        f"block {block}\nstream {stream}\nupload {upload}\nrepeat {repeat}\nflags {flags}\n")
    (tmp_path / "src.bin").write_bytes(b"".join(np.ascontiguousarray(s).tobytes() for s in src))
    print(f"C client case {name}", flush=True)
    r = subprocess.run([exe, str(tmp_path / "case.txt"), str(tmp_path / "src.bin"), str(tmp_path / "dst.bin")],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", f"{name}: rc {r.returncode}\n{r.stdout}\n{r.stderr}"
    got = np.frombuffer((tmp_path / "dst.bin").read_bytes(), dtype=np.uint8)
    assert got.size == sum(w.nbytes for w in want)
    off = 0
    for k, w in enumerate(want):
        wb = np.ascontiguousarray(w).view(np.uint8).ravel()
        assert np.array_equal(got[off:off + wb.size], wb), f"{name}: destination {k} differs from the oracle"
        off += wb.size
