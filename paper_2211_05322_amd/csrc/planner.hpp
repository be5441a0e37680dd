// planner.hpp -- host-side planning of one cross-mesh resharding task.
//
// Steps (all host, no HIP):
//   parse      spec strings -> mesh axes per tensor dimension (Section 2.2)
//   layout     device -> shard index per dimension, shard bounds per dimension
//   tasks      unit tasks = non-empty intersections of a source shard and a
//              destination shard, with all owners and all receivers
//              (Section 2.2; the same slices as the appendix cut-point
//              decomposition, computed here dimension by dimension as
//              intersections of shard intervals)
//   senders    one owner per task: naive (lowest index) or longest-first
//              greedy balancing of sent bytes (Section 3.2, Eq. 4)
//   lowering   each task -> pieces (collapsed strided boxes) -> chunks
//              (descriptors, one per workgroup)
#pragma once

#include <atomic>
#include <cstdint>
#include <mutex>
#include <string>
#include <vector>

#include "desc.h"

namespace rs {

struct Layout {
    std::vector<int64_t> mesh;               // mesh shape
    std::vector<std::vector<int>> axes;      // per tensor dim: mesh axes, major to minor
    std::vector<int64_t> nshards;            // per tensor dim
    std::vector<std::vector<int64_t>> bounds;  // per dim: nshards+1 cut positions
    int64_t ndev = 0;
    std::vector<int64_t> dev_shard;          // [dev * ndim + dim] -> shard index
    std::vector<int64_t> shard_devs_off;     // CSR over linearised shard tuples
    std::vector<int32_t> shard_devs;         //   -> devices holding that shard (ascending)
};

struct UnitTask {
    std::vector<int64_t> lo, hi;   // slice of D
    int64_t src_shard = 0;         // linearised source shard tuple
    int64_t dst_shard = 0;         // linearised destination shard tuple
    int64_t bytes = 0;
    int32_t sender = -1;           // chosen owner
};

struct Tuning {
    int64_t chunk_bytes = 0;   // 0: automatic
    int32_t block_threads = 256;
    bool block_is_default = true;  // the caller left the block size to the library
    int32_t max_wgs_per_cu = 0;  // the caller's cap (0: none)
    bool cap_is_default = true;  // the caller left the cap to the library (chosen at launch)
    int32_t gather_band = 0;     // row gather: segments per column band (0: whole rows)
};

// A number no other plan of this process has (plans are told apart by it,
// not by address, which a later plan may reuse).
inline uint64_t next_plan_serial() {
    static std::atomic<uint64_t> n{0};
    return ++n;
}

struct Plan {
    const uint64_t serial = next_plan_serial();
    int ndim = 0;
    std::vector<int64_t> shape;
    int64_t es = 0;            // element size in bytes
    unsigned flags = 0;
    Tuning tuning;
    Layout src, dst;
    // Local layouts: dimension k of a device's buffer is tensor dimension
    // perm[k] (identity unless the caller permuted a side).
    std::vector<int> sperm, dperm;
    std::vector<UnitTask> tasks;
    std::vector<Desc> descs;
    std::vector<int32_t> fan;  // receiver lists, referenced by Desc::fan_off/nfan
    int64_t bytes_read = 0, bytes_written = 0, max_fanout = 0;
    int64_t align = 1;         // required buffer alignment in bytes
    bool too_many = false;     // lowering stopped: descriptor table over its cap
    bool tile_span_too_long = false;  // lowering stopped: one transpose tile spans 2^32 bytes or more
    uint32_t lds_bytes = 0;    // LDS the realignment chunks need per workgroup
    size_t n_direct = 0;       // descs[0, n_direct): direct chunks
    size_t n_gather = 0;       // descs[n_direct, n_direct + n_gather): row-gather chunks;
    size_t n_gather_u = 0;     // then n_gather_u unaligned row-gather chunks (the last n_unit
    size_t n_unit = 0;         // of them unit-gather chunks, their own kernel);
    size_t n_transpose = 0;    // then n_transpose tile-transpose chunks;
    uint32_t transpose_rows = 0;  // rows of the widest transpose tile (LDS: rows x 128 bytes)
                               // the rest: realignment chunks
    std::vector<Seg> segs;     // row-gather segment entries
    int64_t gather_fanout = 0; // largest receiver count among row-gather chunks
    int64_t gather_u_fanout = 0; // ... among unaligned row-gather chunks
    int64_t gather_u_segs = 0;   // most segments per row among unaligned row-gather groups
    uint64_t gather_u_bytes = 0; // destination bytes of the slot chunks, and their nominal
    uint64_t gather_u_room = 0;  //     capacity (chunks x chunk size): how full they are
    bool gather_u_short = false; // some slot group has segments under 16 bytes
    int64_t unit_fanout = 0;     // ... and among the unit-gather groups:
    int64_t unit_segs = 0;       //     receivers, segments per row
    int64_t direct_fanout = 0; // largest receiver count among direct chunks
    size_t n_phase1 = 0;       // descs[0, n_phase1) run before descs[n_phase1, n_direct)
                               // (two launches; only the all-gather strategy has a second phase)
    std::vector<int64_t> src_local_numel, dst_local_numel;  // per device

    // Device copy of [descs | fan], uploaded on the first execute on each HIP
    // device (index = device ordinal).
    static constexpr int kMaxHipDevices = 64;
    mutable std::mutex mu;
    mutable void *d_table[kMaxHipDevices] = {};
};

// Returns "" on success, else an error message; `code` receives the status.
std::string parse_spec(const char *spec, int ndim, int mesh_ndim, std::vector<std::vector<int>> &axes);
std::string build_layout(const std::vector<int64_t> &shape, const std::vector<int64_t> &mesh,
                         const std::vector<std::vector<int>> &axes, Layout &out);
void build_tasks(Plan &p);
void choose_senders(Plan &p);
void lower(Plan &p);

// Local (per-device) shape on one side.
void local_shape(const Plan &p, int side, int64_t dev, int64_t *out);

}  // namespace rs
