"""Thin Python binding of libreshard.so (ctypes; argument marshalling only).

The names mirror the C ABI in include/reshard.h.  Buffers are passed as raw
pointers (ints) or torch tensors (their data_ptr()); streams as a
torch.cuda.Stream, a raw hipStream_t int, or None for the current torch
stream.  All data movement happens inside the library's HIP kernel; this
module never copies tensor data.  If the library is missing it raises --
there is no fallback.
"""

from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libreshard.so")

RESHARD_OK, RESHARD_EINVAL, RESHARD_EUNSUPPORTED, RESHARD_ENOMEM, RESHARD_EHIP = range(5)
RESHARD_SENDER_NAIVE = 0x1
RESHARD_XCD_REMAP = 0x2
RESHARD_TASK_ORDER = 0x4
RESHARD_NO_REALIGN = 0x8
RESHARD_LDS_STAGING = 0x10
RESHARD_STRATEGY_SENDRECV = 0x20
RESHARD_STRATEGY_ALLGATHER = 0x40
RESHARD_NO_GATHER = 0x100
RESHARD_MAX_BUFFERS = 496

_DTYPES = {"uint8": 0, "int8": 1, "float16": 2, "bfloat16": 3, "float32": 4, "int32": 5,
           "float64": 6, "int64": 7, "uint16": 8, "int16": 9, "uint32": 10, "uint64": 11}

_STATUS = {RESHARD_EINVAL: "EINVAL", RESHARD_EUNSUPPORTED: "EUNSUPPORTED",
           RESHARD_ENOMEM: "ENOMEM", RESHARD_EHIP: "EHIP"}


class ReshardError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


class reshard_tuning_t(ctypes.Structure):
    _fields_ = [("chunk_bytes", ctypes.c_int64), ("block_threads", ctypes.c_int32),
                ("max_wgs_per_cu", ctypes.c_int32), ("gather_band", ctypes.c_int32),
                ("reserved", ctypes.c_int32 * 3)]


_lib = None
_I64P = ctypes.POINTER(ctypes.c_int64)
_VPP = ctypes.POINTER(ctypes.c_void_p)


def load(path=None):
    """Load libreshard.so (built by paper_2211_05322_amd.build); raise if it is missing."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise ImportError(f"libreshard.so not built at {path}; run `python -m paper_2211_05322_amd.build`")
    # torch first: its HIP runtime (libamdhip64 from its own directory,
    # soname libamdhip64.so.7) then satisfies the library's dependency on
    # libamdhip64.so.7.  Opened the other way round, the process would map
    # the system runtime for the library and torch's for its tensors and
    # streams -- two HIP runtimes, with kernels registered in only one.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    plan_args = [ctypes.c_int, _I64P, ctypes.c_int, ctypes.c_int, _I64P, ctypes.c_char_p,
                 ctypes.c_int, _I64P, ctypes.c_char_p, ctypes.c_uint]
    lib.reshard_plan.argtypes = plan_args + [ctypes.POINTER(ctypes.c_void_p)]
    lib.reshard_plan.restype = ctypes.c_int
    lib.reshard_plan_ex.argtypes = plan_args + [ctypes.POINTER(reshard_tuning_t), ctypes.POINTER(ctypes.c_void_p)]
    _I32P = ctypes.POINTER(ctypes.c_int32)
    lib.reshard_plan_permuted.argtypes = [ctypes.c_int, _I64P, ctypes.c_int, ctypes.c_int, _I64P, ctypes.c_char_p,
                                          _I32P, ctypes.c_int, _I64P, ctypes.c_char_p, _I32P, ctypes.c_uint,
                                          ctypes.POINTER(reshard_tuning_t), ctypes.POINTER(ctypes.c_void_p)]
    lib.reshard_plan_permuted.restype = ctypes.c_int
    lib.reshard_plan_unit_gather_chunks.argtypes = [ctypes.c_void_p]
    lib.reshard_plan_unit_gather_chunks.restype = ctypes.c_int64
    lib.reshard_plan_transpose_chunks.argtypes = [ctypes.c_void_p]
    lib.reshard_plan_transpose_chunks.restype = ctypes.c_int64
    lib.reshard_plan_ex.restype = ctypes.c_int
    lib.reshard_execute.argtypes = [ctypes.c_void_p, _VPP, _VPP, ctypes.c_void_p]
    lib.reshard_execute.restype = ctypes.c_int
    lib.reshard_execute_noalloc.argtypes = [ctypes.c_void_p, _VPP, _VPP, ctypes.c_void_p]
    lib.reshard_execute_noalloc.restype = ctypes.c_int
    lib.reshard_plan_destroy.argtypes = [ctypes.c_void_p]
    lib.reshard_plan_destroy.restype = None
    lib.reshard_plan_local_shape.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, _I64P]
    lib.reshard_plan_local_shape.restype = ctypes.c_int
    lib.reshard_plan_stats.argtypes = [ctypes.c_void_p] + [_I64P] * 5
    lib.reshard_plan_stats.restype = ctypes.c_int
    lib.reshard_plan_alignment.argtypes = [ctypes.c_void_p]
    lib.reshard_plan_alignment.restype = ctypes.c_int64
    lib.reshard_plan_lds_bytes.argtypes = [ctypes.c_void_p]
    lib.reshard_plan_lds_bytes.restype = ctypes.c_int64
    lib.reshard_plan_upload.argtypes = [ctypes.c_void_p]
    lib.reshard_plan_upload.restype = ctypes.c_int
    lib.reshard_plan_gather_chunks.argtypes = [ctypes.c_void_p]
    lib.reshard_plan_gather_chunks.restype = ctypes.c_int64
    lib.reshard_plan_realign_chunks.argtypes = [ctypes.c_void_p]
    lib.reshard_plan_realign_chunks.restype = ctypes.c_int64
    lib.reshard_plan_unaligned_gather_chunks.argtypes = [ctypes.c_void_p]
    lib.reshard_plan_unaligned_gather_chunks.restype = ctypes.c_int64
    lib.reshard_plan_unit_task.argtypes = [ctypes.c_void_p, ctypes.c_int64, _I64P, _I64P, _I64P,
                                           _I64P, ctypes.c_int64, _I64P, _I64P, ctypes.c_int64, _I64P]
    lib.reshard_plan_unit_task.restype = ctypes.c_int
    lib.reshard_debug_execute_host.argtypes = [ctypes.c_void_p, _VPP, _VPP]
    lib.reshard_debug_execute_host.restype = ctypes.c_int
    lib.reshard_schedule.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                     ctypes.c_int64, ctypes.c_int64, ctypes.c_uint64,
                                     _I64P, _I64P, _I64P, _I64P, _I64P]
    lib.reshard_schedule.restype = ctypes.c_int
    lib.reshard_pipeline_simulate.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_double,
                                              ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_int32,
                                              ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32)]
    lib.reshard_pipeline_simulate.restype = ctypes.c_int
    lib.reshard_last_error.argtypes = []
    lib.reshard_last_error.restype = ctypes.c_char_p
    lib.reshard_version.argtypes = []
    lib.reshard_version.restype = ctypes.c_char_p
    if path == LIB_PATH:
        _lib = lib
    return lib


def _check(status):
    if status != RESHARD_OK:
        raise ReshardError(status, load().reshard_last_error().decode())


def _i64(vals):
    vals = [int(v) for v in vals]
    return (ctypes.c_int64 * max(1, len(vals)))(*vals)


def _dtype_code(dtype):
    name = str(dtype).replace("torch.", "")
    if name not in _DTYPES:
        raise ValueError(f"unsupported dtype {dtype}")
    return _DTYPES[name]


def _addr(b):
    if b is None or isinstance(b, int):
        return b
    return b.data_ptr() if b.numel() > 0 else None


def pointer_array(bufs):
    """The `void *const *` array reshard_execute takes, built once.

    `bufs` holds tensors (an empty one passes NULL), integer addresses or
    None.  A caller that reshards the same buffers repeatedly can build the
    two arrays once and pass them to every reshard_execute, which then skips
    the per-buffer marshalling.  The array holds addresses only: the tensors
    must stay alive (and unmoved) while it is in use.
    """
    if isinstance(bufs, ctypes.Array):
        return bufs
    return (ctypes.c_void_p * max(1, len(bufs)))(*[_addr(b) for b in bufs])


_ptrs = pointer_array


class Plan:
    """Owns a reshard_plan_t*; destroyed with the object."""

    def __init__(self, handle, shape, src_mesh, dst_mesh, dtype):
        self._h = ctypes.c_void_p(handle)
        self.shape = tuple(shape)
        self.ndim = len(self.shape)
        self.src_mesh = tuple(src_mesh)
        self.dst_mesh = tuple(dst_mesh)
        self.dtype = dtype
        n = 1
        for m in self.src_mesh:
            n *= m
        self.n_src = n
        n = 1
        for m in self.dst_mesh:
            n *= m
        self.n_dst = n

    @property
    def handle(self):
        return self._h

    def __del__(self):
        if getattr(self, "_h", None) and self._h.value and _lib is not None:
            _lib.reshard_plan_destroy(self._h)
            self._h = ctypes.c_void_p(0)


def reshard_plan(shape, dtype, src_mesh, src_spec, dst_mesh, dst_spec, flags=0,
                 chunk_bytes=0, block_threads=0, max_wgs_per_cu=0, gather_band=0, src_perm=None, dst_perm=None):
    """A plan; src_perm / dst_perm (tuples or None) permute each side's local
    buffer layout (buffer dimension k is tensor dimension perm[k])."""
    lib = load()
    h = ctypes.c_void_p()
    args = [len(shape), _i64(shape), _dtype_code(dtype), len(src_mesh), _i64(src_mesh),
            src_spec.encode(), len(dst_mesh), _i64(dst_mesh), dst_spec.encode(), int(flags)]
    if src_perm is not None or dst_perm is not None:
        def perm(p):
            return None if p is None else (ctypes.c_int32 * max(1, len(p)))(*[int(a) for a in p])
        t = reshard_tuning_t(chunk_bytes=int(chunk_bytes), block_threads=int(block_threads),
                             max_wgs_per_cu=int(max_wgs_per_cu), gather_band=int(gather_band))
        _check(lib.reshard_plan_permuted(len(shape), _i64(shape), _dtype_code(dtype), len(src_mesh), _i64(src_mesh),
                                         src_spec.encode(), perm(src_perm), len(dst_mesh), _i64(dst_mesh),
                                         dst_spec.encode(), perm(dst_perm), int(flags), ctypes.byref(t),
                                         ctypes.byref(h)))
    elif chunk_bytes or block_threads or max_wgs_per_cu or gather_band:
        t = reshard_tuning_t(chunk_bytes=int(chunk_bytes), block_threads=int(block_threads),
                             max_wgs_per_cu=int(max_wgs_per_cu), gather_band=int(gather_band))
        _check(lib.reshard_plan_ex(*args, ctypes.byref(t), ctypes.byref(h)))
    else:
        _check(lib.reshard_plan(*args, ctypes.byref(h)))
    return Plan(h.value, shape, src_mesh, dst_mesh, dtype)


def _stream_handle(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def reshard_plan_upload(plan):
    """Upload the plan's tables to the current device (then execute is graph-capturable)."""
    _check(load().reshard_plan_upload(plan.handle))


def reshard_execute(plan, src_bufs, dst_bufs, stream=None):
    """Enqueue the reshard kernel on `stream` (default: torch's current stream).

    `src_bufs` / `dst_bufs`: one buffer per device (tensors, addresses or
    None), or arrays from `pointer_array`.
    """
    if len(src_bufs) != plan.n_src or len(dst_bufs) != plan.n_dst:
        raise ValueError(f"need {plan.n_src} source and {plan.n_dst} destination buffers")
    _check(load().reshard_execute(plan.handle, _ptrs(src_bufs), _ptrs(dst_bufs),
                                  ctypes.c_void_p(_stream_handle(stream))))


def reshard_execute_noalloc(plan, src_bufs, dst_bufs, stream=None):
    """reshard_execute that allocates nothing: the plan's tables go to the
    library's fixed per-device scratch array (see the header for its limit
    and for calls that overlap)."""
    if len(src_bufs) != plan.n_src or len(dst_bufs) != plan.n_dst:
        raise ValueError(f"need {plan.n_src} source and {plan.n_dst} destination buffers")
    _check(load().reshard_execute_noalloc(plan.handle, _ptrs(src_bufs), _ptrs(dst_bufs),
                                          ctypes.c_void_p(_stream_handle(stream))))


def reshard_debug_execute_host(plan, src_bufs, dst_bufs):
    """Run the descriptor table on host buffers (numpy arrays or CPU tensors)."""
    def ptr(b):
        if b is None:
            return None
        if hasattr(b, "ctypes"):
            return b.ctypes.data if b.size > 0 else None
        return b.data_ptr() if b.numel() > 0 else None
    if len(src_bufs) != plan.n_src or len(dst_bufs) != plan.n_dst:
        raise ValueError(f"need {plan.n_src} source and {plan.n_dst} destination buffers")
    _check(load().reshard_debug_execute_host(plan.handle, _ptrs([ptr(b) for b in src_bufs]),
                                             _ptrs([ptr(b) for b in dst_bufs])))


def reshard_plan_local_shape(plan, side, device):
    out = (ctypes.c_int64 * plan.ndim)()
    _check(load().reshard_plan_local_shape(plan.handle, int(side), int(device), out))
    return tuple(out)


def reshard_plan_stats(plan):
    vals = [ctypes.c_int64() for _ in range(5)]
    _check(load().reshard_plan_stats(plan.handle, *[ctypes.byref(v) for v in vals]))
    keys = ("bytes_read", "bytes_written", "n_unit_tasks", "n_descriptors", "max_fanout")
    return {k: v.value for k, v in zip(keys, vals)}


def reshard_plan_alignment(plan):
    return int(load().reshard_plan_alignment(plan.handle))


def reshard_plan_lds_bytes(plan):
    return int(load().reshard_plan_lds_bytes(plan.handle))


def reshard_plan_gather_chunks(plan):
    return int(load().reshard_plan_gather_chunks(plan.handle))


def reshard_plan_realign_chunks(plan):
    return int(load().reshard_plan_realign_chunks(plan.handle))


def reshard_plan_unit_gather_chunks(plan):
    return load().reshard_plan_unit_gather_chunks(plan.handle)


def reshard_plan_transpose_chunks(plan):
    return load().reshard_plan_transpose_chunks(plan.handle)


def reshard_plan_unaligned_gather_chunks(plan):
    return int(load().reshard_plan_unaligned_gather_chunks(plan.handle))


def reshard_plan_unit_task(plan, index):
    lo = (ctypes.c_int64 * plan.ndim)()
    hi = (ctypes.c_int64 * plan.ndim)()
    chosen = ctypes.c_int64()
    snd = (ctypes.c_int64 * plan.n_src)()
    rcv = (ctypes.c_int64 * plan.n_dst)()
    ns, nr = ctypes.c_int64(), ctypes.c_int64()
    _check(load().reshard_plan_unit_task(plan.handle, int(index), lo, hi, ctypes.byref(chosen),
                                         snd, plan.n_src, ctypes.byref(ns), rcv, plan.n_dst,
                                         ctypes.byref(nr)))
    return {"box": tuple(zip(tuple(lo), tuple(hi))), "sender": chosen.value,
            "senders": list(snd[:ns.value]), "receivers": list(rcv[:nr.value])}


SCHED_ALGOS = {"naive": 0, "load_balance": 1, "dfs": 2, "randomized": 3, "ensemble": 4}


def reshard_schedule(plan, src_devices_per_host, dst_devices_per_host, algo="ensemble",
                     max_dfs_nodes=200000, random_rounds=16, seed=0):
    """Sender choice and start times under the multi-host model (host-side only)."""
    n = reshard_plan_stats(plan)["n_unit_tasks"]
    snd = (ctypes.c_int64 * max(1, n))()
    st = (ctypes.c_int64 * max(1, n))()
    mk, lb, nodes = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(load().reshard_schedule(plan.handle, int(src_devices_per_host), int(dst_devices_per_host),
                                   SCHED_ALGOS[algo], int(max_dfs_nodes), int(random_rounds), int(seed),
                                   snd, st, ctypes.byref(mk), ctypes.byref(lb), ctypes.byref(nodes)))
    return {"senders": list(snd[:n]), "starts": list(st[:n]), "makespan": mk.value,
            "lower_bound": lb.value, "dfs_nodes": nodes.value}


def reshard_pipeline_simulate(stages, microbatches, eager, t_fwd, t_bwd, t_comm_fwd, t_comm_bwd=None,
                              serial_links=True):
    """(latency, per-stage peak live micro-batches) of one pipelined iteration."""
    lat = ctypes.c_double()
    peak = (ctypes.c_int32 * max(1, int(stages)))()
    _check(load().reshard_pipeline_simulate(int(stages), int(microbatches), int(bool(eager)), float(t_fwd),
                                            float(t_bwd), float(t_comm_fwd),
                                            float(t_comm_fwd if t_comm_bwd is None else t_comm_bwd),
                                            int(bool(serial_links)), ctypes.byref(lat), peak))
    return lat.value, list(peak[:int(stages)])


def reshard_last_error():
    return load().reshard_last_error().decode()


def reshard_version():
    return load().reshard_version().decode()


# ------------------------------------------------------------ conveniences

def local_shapes(plan, side):
    n = plan.n_src if side == 0 else plan.n_dst
    return [reshard_plan_local_shape(plan, side, k) for k in range(n)]


def empty_shards(plan, side, device="cuda"):
    """Allocate one dense buffer per device of one side (torch, no data movement)."""
    import torch
    dt = getattr(torch, str(plan.dtype).replace("torch.", ""))
    return [torch.empty(s, dtype=dt, device=device) for s in local_shapes(plan, side)]
