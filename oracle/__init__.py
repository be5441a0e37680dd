"""CPU oracle for cross-mesh resharding -- TEST INFRASTRUCTURE ONLY.

This package is the plain, slow, obviously correct definition of what a
cross-mesh resharding task produces, written in numpy from the paper
("On Optimizing the Communication of Model Parallelism", Zhuang et al.,
MLSys 2023).  It shares no code with the HIP path and imports nothing from
it.  Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may import it; the product path never does.

Parity status of every function is stated in :mod:`oracle.reshard`.
"""

from .reshard import (  # noqa: F401
    parse_spec,
    split_bounds,
    device_coords,
    shard_index,
    device_box,
    local_shape,
    shard,
    unshard,
    reshard,
    unit_tasks,
    choose_senders_naive,
    choose_senders_lpt,
    traffic_bytes,
)
