"""Synthetic workloads and seeded input generators.

This module holds data only: the resharding workloads (tensor shape, element
type, value distribution, the two meshes and their sharding specs) and the
seeded generators of the logical tensor.  It contains none of the resharding
arithmetic, so both the HIP path and the CPU oracle can be fed from it.

The five workloads stand in for the tensors the paper reshards: a small 2-D
fp32 tensor, the GPT layer activation (batch 8, sequence 1024, hidden 4096,
Section 5.2 and Table 4), a 16x2048x5120 fp16 tensor fanned out to a fully
replicated mesh, the U-Transformer skip tensor with an uneven split of H=66
into four, and a GPT-3-width (hidden 12288, Table 1) activation with 4x
replication on the destination.  Values are drawn from a seeded generator;
the copy is bit-exact so the distribution only matters for realism.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    shape: tuple
    dtype: str            # "float32", "float16", ...
    dist: str             # "uniform" (U[-1,1)), "normal" (N(0,1)), "iota", "bits"
    src_mesh: tuple
    src_spec: str
    dst_mesh: tuple
    dst_spec: str
    src_perm: tuple = None  # buffer dimension order of each side (None: tensor order)
    dst_perm: tuple = None

    @property
    def itemsize(self):
        return torch.empty((), dtype=getattr(torch, self.dtype)).element_size()

    @property
    def numel(self):
        n = 1
        for s in self.shape:
            n *= s
        return n


WORKLOADS = {
    1: Workload("fp32_256x1024_mesh1x2_to_2x2", (256, 1024), "float32", "uniform",
                (1, 2), "S^1 R", (2, 2), "R S^0"),
    2: Workload("gpt_act_fp16_8x1024x4096_batch_to_seq", (8, 1024, 4096), "float16", "normal",
                (2, 4), "S^0 R S^1", (2, 4), "R S^0 S^1"),
    3: Workload("fp16_16x2048x5120_s01_to_replicated", (16, 2048, 5120), "float16", "normal",
                (2, 4), "R R S^{01}", (2, 4), "R R R"),
    4: Workload("utrans_skip_fp16_32x512x66x64_to_H4", (32, 512, 66, 64), "float16", "normal",
                (2, 2), "S^0 S^1 R R", (4, 2), "R R S^0 R"),
    5: Workload("gpt3_act_fp16_8x2048x12288_hidden32_to_seq8x4rep", (8, 2048, 12288), "float16",
                "normal", (4, 8), "R R S^{01}", (4, 8), "R S^1 R"),
}

# The resharding the benchmark times: the largest tensor (403 MB, 2.01 GB moved).
BENCH_WORKLOAD = 5

# Workloads 5 and 3 with a last dimension that the shard count does not
# divide: the balanced split gives segments of two widths whose rows sit in
# different 16-byte phases on the two sides (the unaligned row-gather path);
# and misaligned rows that reach their destination in runs.
UNEVEN_WORKLOADS = {
    "uneven5": Workload("gpt3_act_fp16_8x2048x12300_hidden32_uneven_to_seq8x4rep", (8, 2048, 12300), "float16",
                        "normal", (4, 8), "R R S^{01}", (4, 8), "R S^1 R"),
    "uneven3": Workload("fp16_16x2048x5130_s01_uneven_to_replicated", (16, 2048, 5130), "float16", "normal",
                        (2, 4), "R R S^{01}", (2, 4), "R R R"),
    # uneven workload 5 to one replica: 32 senders per destination row at
    # fan-out 1 (the unit gather)
    "uneven5_1rep": Workload("gpt3_act_fp16_8x2048x12300_hidden32_uneven_to_seq8_1rep", (8, 2048, 12300), "float16",
                             "normal", (4, 8), "R R S^{01}", (1, 8), "R S^1 R"),
    # the middle dimension split 1024/1023 on the source and the outer one on
    # the destination, with 24602-byte rows: destination rows contiguous only
    # in runs of 1024 or 1023, in different 16-byte phases; fan-out 1, 2, 4
    "runs1": Workload("fp16_8x2047x12301_mid_to_outer_runs_1rep", (8, 2047, 12301), "float16", "normal",
                      (2,), "R S^0 R", (2,), "S^0 R R"),
    "runs2": Workload("fp16_8x2047x12301_mid_to_outer_runs_2rep", (8, 2047, 12301), "float16", "normal",
                      (2,), "R S^0 R", (2, 2), "S^0 R R"),
    "runs4": Workload("fp16_8x2047x12301_mid_to_outer_runs_4rep", (8, 2047, 12301), "float16", "normal",
                      (2,), "R S^0 R", (2, 4), "S^0 R R"),
}


# Reshards that also change the buffers' dimension order (the paper's specs
# never do): the GPT activation stored [batch, hidden, seq] on the
# destination, and the GPT-3-width one likewise with 4x replication.  Each
# task is a tile transpose.
TRANSPOSED_WORKLOADS = {
    "transposed2": Workload("gpt_act_fp16_8x1024x4096_batch_to_seq_hidden_major", (8, 1024, 4096), "float16",
                            "normal", (2, 4), "S^0 R S^1", (2, 4), "R S^0 S^1", None, (0, 2, 1)),
    "transposed5": Workload("gpt3_act_fp16_8x2048x12288_hidden32_to_seq8x4rep_hidden_major", (8, 2048, 12288),
                            "float16", "normal", (4, 8), "R R S^{01}", (4, 8), "R S^1 R", None, (0, 2, 1)),
}


# The multi-to-multi microbenchmark of the paper's Table 3: tensor
# (1024, 1024, 512), (case, send spec, recv spec, send mesh, recv mesh); a
# mesh row is one node.  Table 3 prints case 1's send mesh as "(2.4)" and case
# 5's receive spec as "S_{0}RR"; they are read as (2,4) and S^0RR.
TABLE3_SHAPE = (1024, 1024, 512)
TABLE3_CASES = [
    (1, "S^0RR", "S^0RR", (2, 4), (2, 4)),
    (2, "RRR", "S^0RR", (2, 4), (2, 4)),
    (3, "RS^0R", "S^0RR", (2, 4), (2, 4)),
    (4, "RS^{01}R", "S^{01}RR", (2, 4), (2, 4)),
    (5, "S^1RR", "S^0RR", (2, 4), (2, 4)),
    (6, "S^0RR", "S^0RR", (2, 4), (3, 4)),
    (7, "S^1RR", "RRR", (1, 4), (2, 4)),
    (8, "RRR", "RRR", (2, 3), (3, 2)),
    (9, "RS^0R", "RRS^0", (2, 4), (2, 4)),
]


def fanout_workload(receivers, nbytes=1 << 30):
    """One sender to `receivers` devices, fully replicated on both sides.

    The shape of the paper's single-sender microbenchmark (Section 5.1.1: a
    1 GB message from one GPU to 1..4 GPUs, replicated specs), as fp16.
    """
    return Workload(f"replicate_fp16_{nbytes >> 20}MiB_1to{receivers}", (nbytes // 2,), "float16", "normal",
                    (1,), "R", (receivers,), "R")


def workload_by_name(key):
    """WORKLOADS id (1..5 or "1".."5"), an UNEVEN_WORKLOADS or TRANSPOSED_WORKLOADS key, or "fanoutR"
    (R receivers, 1 GiB)."""
    key = str(key)
    if key.startswith("fanout"):
        return fanout_workload(int(key[len("fanout"):]))
    if key in UNEVEN_WORKLOADS:
        return UNEVEN_WORKLOADS[key]
    if key in TRANSPOSED_WORKLOADS:
        return TRANSPOSED_WORKLOADS[key]
    return WORKLOADS[int(key)]


def make_tensor(shape, dtype, dist, seed, device="cpu"):
    """Seeded logical tensor of the given shape/dtype/distribution.

    * ``uniform``: U[-1, 1) drawn in float32, then cast.
    * ``normal``:  N(0, 1) drawn in float32, then cast (round to nearest even).
    * ``iota``:    element bits = row-major linear index modulo 2^(8*itemsize),
                   so a misplaced element names where it came from.
    * ``bits``:    uniformly random bit patterns (NaNs, infinities, -0 included).
    On CUDA devices the torch CUDA generator is used, so values differ from the
    CPU stream of the same seed; each side of a comparison must use one device.
    """
    tdt = getattr(torch, dtype)
    shape = tuple(int(s) for s in shape)
    if device == "cpu":
        g = torch.Generator(device="cpu").manual_seed(seed)
    else:
        g = torch.Generator(device=device).manual_seed(seed)
    if dist == "uniform":
        return (torch.rand(shape, generator=g, device=device, dtype=torch.float32) * 2 - 1).to(tdt)
    if dist == "normal":
        return torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(tdt)
    itemsize = torch.empty((), dtype=tdt).element_size()
    bits_dt = {1: torch.uint8, 2: torch.int16, 4: torch.int32, 8: torch.int64}[itemsize]
    n = 1
    for s in shape:
        n *= s
    if dist == "iota":
        width = 8 * itemsize
        idx = torch.arange(n, dtype=torch.int64, device=device)
        if width < 64:
            idx = idx & ((1 << width) - 1)
            if width > 8:
                idx = torch.where(idx >= (1 << (width - 1)), idx - (1 << width), idx)
        return idx.to(bits_dt).view(tdt).reshape(shape)
    if dist == "bits":
        raw = torch.randint(0, 256, (n * itemsize,), generator=g, device=device, dtype=torch.uint8)
        return raw.view(bits_dt).view(tdt).reshape(shape)
    raise ValueError(f"unknown distribution {dist!r}")


def make_workload_tensor(w: Workload, seed=0, device="cpu", dist=None):
    return make_tensor(w.shape, w.dtype, dist or w.dist, seed, device)


def as_numpy_bits(t: torch.Tensor) -> np.ndarray:
    """Host numpy view of a tensor's raw bits (unsigned ints of its element size)."""
    t = t.detach().contiguous().cpu()
    it = t.element_size()
    dt = {1: torch.uint8, 2: torch.int16, 4: torch.int32, 8: torch.int64}[it]
    return t.view(dt).numpy().view(f"u{it}")
