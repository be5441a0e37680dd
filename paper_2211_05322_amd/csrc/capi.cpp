// capi.cpp -- C ABI of libreshard.so: planning, queries, host interpreter.
// reshard_execute and the kernels live in execute.hip.
#include <algorithm>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/reshard.h"
#include "planner.hpp"
#include "status.hpp"

namespace rs {
// Defined in execute.hip: frees the plan's device table (if any).
void release_device_table(const Plan &p);

thread_local std::string g_last_error;

reshard_status_t fail(reshard_status_t st, const std::string &msg) noexcept {
    try {
        g_last_error = msg;
    } catch (...) {
        g_last_error.clear();
    }
    return st;
}

reshard_status_t fail(reshard_status_t st, const char *msg) noexcept {
    try {
        g_last_error = msg;
    } catch (...) {
        g_last_error.clear();
    }
    return st;
}
}  // namespace rs

using rs::fail;

namespace {

int64_t elem_size(reshard_dtype_t dt) {
    switch (dt) {
        case RESHARD_U8: case RESHARD_I8: return 1;
        case RESHARD_F16: case RESHARD_BF16: case RESHARD_U16: case RESHARD_I16: return 2;
        case RESHARD_F32: case RESHARD_I32: case RESHARD_U32: return 4;
        case RESHARD_F64: case RESHARD_I64: case RESHARD_U64: return 8;
    }
    return 0;
}

bool mul_ok(int64_t a, int64_t b, int64_t limit, int64_t &out) {
    if (a != 0 && b > limit / a) return false;
    out = a * b;
    return true;
}

reshard_status_t check_mesh(const char *side, int mesh_ndim, const int64_t *mesh, int64_t &ndev) {
    if (mesh_ndim < 1 || mesh_ndim > RESHARD_MAX_MESH_NDIM)
        return fail(RESHARD_EINVAL, std::string(side) + " mesh must have 1..8 axes, got " + std::to_string(mesh_ndim));
    if (!mesh) return fail(RESHARD_EINVAL, std::string(side) + " mesh pointer is NULL");
    ndev = 1;
    for (int i = 0; i < mesh_ndim; ++i) {
        if (mesh[i] < 1)
            return fail(RESHARD_EINVAL, std::string(side) + " mesh axis " + std::to_string(i) + " is " +
                                            std::to_string(mesh[i]) + "; must be >= 1");
        if (!mul_ok(ndev, mesh[i], RESHARD_MAX_BUFFERS, ndev))
            return fail(RESHARD_EUNSUPPORTED, std::string(side) + " mesh has more than " +
                                                  std::to_string(RESHARD_MAX_BUFFERS) + " devices");
    }
    return RESHARD_OK;
}

// A layout permutation: NULL (identity) or an ordering of 0..ndim-1.
reshard_status_t check_perm(const char *side, const int32_t *perm, int ndim, std::vector<int> &out) {
    out.resize(size_t(ndim));
    std::vector<char> seen(size_t(ndim), 0);
    for (int k = 0; k < ndim; ++k) {
        const int a = perm ? int(perm[k]) : k;
        if (a < 0 || a >= ndim || seen[size_t(a)])
            return fail(RESHARD_EINVAL, std::string(side) + " permutation is not an ordering of the " +
                                            std::to_string(ndim) + " tensor dimensions");
        seen[size_t(a)] = 1;
        out[size_t(k)] = a;
    }
    return RESHARD_OK;
}

reshard_status_t make_plan(int ndim, const int64_t *shape, reshard_dtype_t dtype, int smn, const int64_t *sm,
                           const char *sspec, int dmn, const int64_t *dm, const char *dspec, unsigned flags,
                           const reshard_tuning_t *tuning, reshard_plan_t **out, const int32_t *sperm = nullptr,
                           const int32_t *dperm = nullptr) {
    if (!out) return fail(RESHARD_EINVAL, "out is NULL");
    *out = nullptr;
    if (ndim < 1 || ndim > RESHARD_MAX_NDIM)
        return fail(RESHARD_EINVAL, "ndim must be 1..8, got " + std::to_string(ndim));
    if (!shape) return fail(RESHARD_EINVAL, "shape is NULL");
    const int64_t es = elem_size(dtype);
    if (es == 0) return fail(RESHARD_EINVAL, "unknown dtype " + std::to_string(int(dtype)));
    int64_t total = es;
    for (int i = 0; i < ndim; ++i) {
        if (shape[i] < 0) return fail(RESHARD_EINVAL, "shape[" + std::to_string(i) + "] is negative");
        if (!mul_ok(total, shape[i], int64_t(1) << 56, total))
            return fail(RESHARD_EUNSUPPORTED, "tensor larger than 2^56 bytes");
    }
    if (flags & ~(RESHARD_SENDER_NAIVE | RESHARD_XCD_REMAP | RESHARD_TASK_ORDER | RESHARD_NO_REALIGN |
                  RESHARD_LDS_STAGING | RESHARD_STRATEGY_SENDRECV | RESHARD_STRATEGY_ALLGATHER | RESHARD_NO_GATHER))
        return fail(RESHARD_EINVAL, "unknown flag bits");
    if ((flags & RESHARD_STRATEGY_SENDRECV) && (flags & RESHARD_STRATEGY_ALLGATHER))
        return fail(RESHARD_EINVAL, "at most one strategy flag");
    rs::Tuning tn;
    if (tuning) {
        for (int r : tuning->reserved)
            if (r != 0) return fail(RESHARD_EINVAL, "tuning.reserved must be zero");
        if (tuning->chunk_bytes < 0) return fail(RESHARD_EINVAL, "tuning.chunk_bytes is negative");
        const int bt = tuning->block_threads;
        if (bt != 0 && bt != 64 && bt != 128 && bt != 256 && bt != 512 && bt != 1024)
            return fail(RESHARD_EINVAL, "tuning.block_threads must be 64, 128, 256, 512 or 1024");
        const int cap = tuning->max_wgs_per_cu;
        if (cap != 0 && cap != -1 && (cap < 2 || cap > 32))
            return fail(RESHARD_EINVAL, "tuning.max_wgs_per_cu must be -1, 0 or 2..32");
        tn.chunk_bytes = tuning->chunk_bytes;
        if (bt) {
            tn.block_threads = bt;
            tn.block_is_default = false;
        }
        tn.max_wgs_per_cu = cap;
        if (tuning->gather_band < 0) return fail(RESHARD_EINVAL, "tuning.gather_band is negative");
        tn.gather_band = tuning->gather_band;
    }
    // 0: the library picks each kernel's residency at launch from its
    // fan-out; -1: no cap
    tn.cap_is_default = tn.max_wgs_per_cu == 0;
    if (tn.max_wgs_per_cu == -1) tn.max_wgs_per_cu = 0;
    int64_t ns = 0, nd = 0;
    reshard_status_t st = check_mesh("source", smn, sm, ns);
    if (st != RESHARD_OK) return st;
    st = check_mesh("destination", dmn, dm, nd);
    if (st != RESHARD_OK) return st;
    if (ns + nd > RESHARD_MAX_BUFFERS)
        return fail(RESHARD_EUNSUPPORTED, "source and destination meshes have " + std::to_string(ns + nd) +
                                              " devices; at most " + std::to_string(RESHARD_MAX_BUFFERS));
    std::vector<std::vector<int>> sax, dax;
    std::string err = rs::parse_spec(sspec, ndim, smn, sax);
    if (!err.empty()) return fail(RESHARD_EINVAL, "source " + err);
    err = rs::parse_spec(dspec, ndim, dmn, dax);
    if (!err.empty()) return fail(RESHARD_EINVAL, "destination " + err);
    std::vector<int> sp, dp;
    st = check_perm("source", sperm, ndim, sp);
    if (st != RESHARD_OK) return st;
    st = check_perm("destination", dperm, ndim, dp);
    if (st != RESHARD_OK) return st;
    bool permuted = false;
    for (int k = 0; k < ndim; ++k) permuted = permuted || sp[size_t(k)] != k || dp[size_t(k)] != k;
    if (permuted && (flags & (RESHARD_STRATEGY_SENDRECV | RESHARD_STRATEGY_ALLGATHER)))
        return fail(RESHARD_EUNSUPPORTED, "the comparison strategies take unpermuted layouts only");

    rs::Plan *p = new (std::nothrow) rs::Plan();
    if (!p) return fail(RESHARD_ENOMEM, "out of host memory");
    try {
        p->ndim = ndim;
        p->shape.assign(shape, shape + ndim);
        p->es = es;
        p->flags = flags;
        p->tuning = tn;
        p->sperm = sp;
        p->dperm = dp;
        rs::build_layout(p->shape, std::vector<int64_t>(sm, sm + smn), sax, p->src);
        rs::build_layout(p->shape, std::vector<int64_t>(dm, dm + dmn), dax, p->dst);
        // bound the number of unit tasks before enumerating them
        int64_t bound = 1;
        for (int d = 0; d < ndim; ++d)
            if (!mul_ok(bound, p->src.nshards[d] + p->dst.nshards[d], int64_t(1) << 24, bound)) {
                delete p;
                return fail(RESHARD_EUNSUPPORTED, "more than 2^24 unit tasks");
            }
        rs::build_tasks(*p);
        rs::choose_senders(*p);
        rs::lower(*p);
        if (p->too_many) {
            delete p;
            return fail(RESHARD_EUNSUPPORTED, "lowering needs more than 2^24 workgroup chunks");
        }
        if (p->tile_span_too_long) {
            delete p;
            return fail(RESHARD_EUNSUPPORTED,
                        "a transpose tile of the permuted layouts would span 2^32 bytes or more of one buffer");
        }
    } catch (const std::bad_alloc &) {
        delete p;
        return fail(RESHARD_ENOMEM, "out of host memory while planning");
    }
    *out = reinterpret_cast<reshard_plan_t *>(p);
    return RESHARD_OK;
}

const rs::Plan *as_plan(const reshard_plan_t *p) { return reinterpret_cast<const rs::Plan *>(p); }

}  // namespace

extern "C" {

reshard_status_t reshard_plan(int ndim, const int64_t *shape, reshard_dtype_t dtype, int src_mesh_ndim,
                              const int64_t *src_mesh, const char *src_spec, int dst_mesh_ndim,
                              const int64_t *dst_mesh, const char *dst_spec, unsigned flags,
                              reshard_plan_t **out) {
    return rs::guarded([&]() -> reshard_status_t {
        return make_plan(ndim, shape, dtype, src_mesh_ndim, src_mesh, src_spec, dst_mesh_ndim, dst_mesh, dst_spec,
                         flags, nullptr, out);
    });
}

reshard_status_t reshard_plan_ex(int ndim, const int64_t *shape, reshard_dtype_t dtype, int src_mesh_ndim,
                                 const int64_t *src_mesh, const char *src_spec, int dst_mesh_ndim,
                                 const int64_t *dst_mesh, const char *dst_spec, unsigned flags,
                                 const reshard_tuning_t *tuning, reshard_plan_t **out) {
    return rs::guarded([&]() -> reshard_status_t {
        return make_plan(ndim, shape, dtype, src_mesh_ndim, src_mesh, src_spec, dst_mesh_ndim, dst_mesh, dst_spec,
                         flags, tuning, out);
    });
}

reshard_status_t reshard_plan_permuted(int ndim, const int64_t *shape, reshard_dtype_t dtype, int src_mesh_ndim,
                                       const int64_t *src_mesh, const char *src_spec, const int32_t *src_perm,
                                       int dst_mesh_ndim, const int64_t *dst_mesh, const char *dst_spec,
                                       const int32_t *dst_perm, unsigned flags, const reshard_tuning_t *tuning,
                                       reshard_plan_t **out) {
    return rs::guarded([&]() -> reshard_status_t {
        return make_plan(ndim, shape, dtype, src_mesh_ndim, src_mesh, src_spec, dst_mesh_ndim, dst_mesh, dst_spec,
                         flags, tuning, out, src_perm, dst_perm);
    });
}

void reshard_plan_destroy(reshard_plan_t *plan) {
    if (!plan) return;
    rs::Plan *p = reinterpret_cast<rs::Plan *>(plan);
    try {
        rs::release_device_table(*p);
    } catch (...) {  // (the lock cannot be taken: nothing else to release)
    }
    delete p;
}

reshard_status_t reshard_plan_local_shape(const reshard_plan_t *plan, int side, int64_t device,
                                          int64_t *shape_out) {
    return rs::guarded([&]() -> reshard_status_t {
        const rs::Plan *p = as_plan(plan);
        if (!p || !shape_out) return fail(RESHARD_EINVAL, "NULL plan or shape_out");
        if (side != 0 && side != 1) return fail(RESHARD_EINVAL, "side must be 0 (source) or 1 (destination)");
        const int64_t n = side == 0 ? p->src.ndev : p->dst.ndev;
        if (device < 0 || device >= n)
            return fail(RESHARD_EINVAL, "device " + std::to_string(device) + " outside 0.." + std::to_string(n - 1));
        rs::local_shape(*p, side, device, shape_out);
        return RESHARD_OK;
    });
}

reshard_status_t reshard_plan_stats(const reshard_plan_t *plan, int64_t *bytes_read, int64_t *bytes_written,
                                    int64_t *n_unit_tasks, int64_t *n_descriptors, int64_t *max_fanout) {
    return rs::guarded([&]() -> reshard_status_t {
        const rs::Plan *p = as_plan(plan);
        if (!p) return fail(RESHARD_EINVAL, "NULL plan");
        if (bytes_read) *bytes_read = p->bytes_read;
        if (bytes_written) *bytes_written = p->bytes_written;
        if (n_unit_tasks) *n_unit_tasks = int64_t(p->tasks.size());
        if (n_descriptors) *n_descriptors = int64_t(p->descs.size());
        if (max_fanout) *max_fanout = p->max_fanout;
        return RESHARD_OK;
    });
}

int64_t reshard_plan_alignment(const reshard_plan_t *plan) {
    const rs::Plan *p = as_plan(plan);
    return p ? p->align : 0;
}

int64_t reshard_plan_lds_bytes(const reshard_plan_t *plan) {
    const rs::Plan *p = as_plan(plan);
    if (!p) return -1;
    return (p->flags & RESHARD_LDS_STAGING) ? int64_t(p->lds_bytes) : 0;
}

int64_t reshard_plan_gather_chunks(const reshard_plan_t *plan) {
    const rs::Plan *p = as_plan(plan);
    return p ? int64_t(p->n_gather) : -1;
}

int64_t reshard_plan_realign_chunks(const reshard_plan_t *plan) {
    const rs::Plan *p = as_plan(plan);
    return p ? int64_t(p->descs.size() - p->n_direct - p->n_gather - p->n_gather_u - p->n_transpose) : -1;
}

int64_t reshard_plan_unit_gather_chunks(const reshard_plan_t *plan) {
    const rs::Plan *p = as_plan(plan);
    return p ? int64_t(p->n_unit) : -1;
}

int64_t reshard_plan_transpose_chunks(const reshard_plan_t *plan) {
    const rs::Plan *p = as_plan(plan);
    return p ? int64_t(p->n_transpose) : -1;
}

int64_t reshard_plan_unaligned_gather_chunks(const reshard_plan_t *plan) {
    const rs::Plan *p = as_plan(plan);
    return p ? int64_t(p->n_gather_u) : -1;
}

reshard_status_t reshard_plan_unit_task(const reshard_plan_t *plan, int64_t index, int64_t *lo, int64_t *hi,
                                        int64_t *chosen_sender, int64_t *senders, int64_t senders_cap,
                                        int64_t *n_senders, int64_t *receivers, int64_t receivers_cap,
                                        int64_t *n_receivers) {
    return rs::guarded([&]() -> reshard_status_t {
        const rs::Plan *p = as_plan(plan);
        if (!p || !lo || !hi) return fail(RESHARD_EINVAL, "NULL plan, lo or hi");
        if (index < 0 || index >= int64_t(p->tasks.size()))
            return fail(RESHARD_EINVAL, "unit task index " + std::to_string(index) + " out of range");
        if ((senders_cap > 0 && !senders) || (receivers_cap > 0 && !receivers) || senders_cap < 0 || receivers_cap < 0)
            return fail(RESHARD_EINVAL, "NULL output array with non-zero capacity");
        const rs::UnitTask &t = p->tasks[size_t(index)];
        for (int d = 0; d < p->ndim; ++d) {
            lo[d] = t.lo[d];
            hi[d] = t.hi[d];
        }
        if (chosen_sender) *chosen_sender = t.sender;
        const int64_t s0 = p->src.shard_devs_off[t.src_shard], s1 = p->src.shard_devs_off[t.src_shard + 1];
        for (int64_t k = s0; k < s1 && k - s0 < senders_cap; ++k) senders[k - s0] = p->src.shard_devs[k];
        if (n_senders) *n_senders = s1 - s0;
        const int64_t r0 = p->dst.shard_devs_off[t.dst_shard], r1 = p->dst.shard_devs_off[t.dst_shard + 1];
        for (int64_t k = r0; k < r1 && k - r0 < receivers_cap; ++k) receivers[k - r0] = p->dst.shard_devs[k];
        if (n_receivers) *n_receivers = r1 - r0;
        return RESHARD_OK;
    });
}

reshard_status_t reshard_debug_execute_host(const reshard_plan_t *plan, void *const *src_ptrs,
                                            void *const *dst_ptrs) {
    return rs::guarded([&]() -> reshard_status_t {
        const rs::Plan *p = as_plan(plan);
        if (!p || !src_ptrs || !dst_ptrs) return fail(RESHARD_EINVAL, "NULL plan or pointer array");
        for (int64_t k = 0; k < p->src.ndev; ++k)
            if (p->src_local_numel[k] > 0 && !src_ptrs[k])
                return fail(RESHARD_EINVAL, "source buffer " + std::to_string(k) + " is NULL but its shard is not empty");
        for (int64_t k = 0; k < p->dst.ndev; ++k)
            if (p->dst_local_numel[k] > 0 && !dst_ptrs[k])
                return fail(RESHARD_EINVAL, "destination buffer " + std::to_string(k) + " is NULL but its shard is not empty");
        std::vector<uint8_t> lds;
        for (size_t di = 0; di < p->descs.size(); ++di) {
            const rs::Desc &d = p->descs[di];
            const uint32_t w = 1u << rs::kind_log2w(d.kind);
            const uint32_t levels = rs::kind_levels(d.kind);
            const size_t t0 = p->n_direct + p->n_gather + p->n_gather_u;
            if (di >= t0 && di < t0 + p->n_transpose) {
                // tile-transpose chunk: the kernel's tile arithmetic and
                // swizzled LDS tile, every access bounds-checked
                const uint32_t es = uint32_t(p->es), te = rs::tile_elems(es), vpe = 16u / es;
                const uint32_t tr = rs::tile_rows(es, d.kind), slots = tr * es / 16u;  // per column
                const bool ald = (d.kind & rs::kTAlignLoad) != 0, ast = (d.kind & rs::kTAlignStore) != 0;
                if ((1u << (d.kind & 0xFu)) != es) return fail(RESHARD_EINVAL, "internal: transpose element size");
                const uint64_t sbytes = uint64_t(p->src_local_numel[d.src_buf] * p->es);
                lds.assign(tr * rs::kTileBytes, 0);
                for (uint32_t t = d.v0; t < d.v1; ++t) {
                    const rs::TileAt at = rs::tile_offsets(d, t, es);
                    const uint32_t na = std::min(te, d.run - at.ta * te), nb = std::min(tr, d.batch - at.tb * tr);
                    for (uint32_t i = 0; i < tr * 8u; ++i) {  // load phase
                        const uint32_t r = i >> 3, c = i & 7u;
                        if (r >= nb) continue;
                        const uint32_t a0 = c * vpe;
                        const uint32_t nv = a0 < na ? std::min(vpe, na - a0) : 0u;
                        uint8_t x[16] = {0};
                        const uint64_t q = d.src_base + uint32_t(at.src + r * d.ss[0] + c * 16u);
                        if (nv == vpe && ald) {
                            if (q % 16 != 0) return fail(RESHARD_EINVAL, "internal: transpose vector load misaligned");
                            if (q + 16 > sbytes) return fail(RESHARD_EINVAL, "internal: transpose load outside its source shard");
                            std::memcpy(x, static_cast<const char *>(src_ptrs[d.src_buf]) + q, 16);
                        } else {
                            for (uint32_t e = 0; e < nv; ++e) {
                                if (q + (e + 1) * es > sbytes) return fail(RESHARD_EINVAL, "internal: transpose load outside its source shard");
                                std::memcpy(x + e * es, static_cast<const char *>(src_ptrs[d.src_buf]) + q + e * es, es);
                            }
                        }
                        const uint32_t o = rs::tile_lds(r, c, 0, es);
                        if (o + 16 > lds.size()) return fail(RESHARD_EINVAL, "internal: transpose LDS write out of range");
                        std::memcpy(lds.data() + o, x, 16);
                    }
                    for (uint32_t i = 0; i < te * slots; ++i) {  // store phase
                        const uint32_t a = i / slots, j = i % slots;
                        if (a >= na) continue;
                        const uint32_t b0 = j * vpe;
                        const uint32_t nv = b0 < nb ? std::min(vpe, nb - b0) : 0u;
                        if (nv == 0) continue;
                        uint8_t y[16] = {0};
                        for (uint32_t e = 0; e < vpe; ++e) {
                            const uint32_t o = rs::tile_lds(b0 + e, (a * es) >> 4, (a * es) & 15u, es);
                            if (o + es > lds.size()) return fail(RESHARD_EINVAL, "internal: transpose LDS read out of range");
                            std::memcpy(y + e * es, lds.data() + o, es);
                        }
                        for (uint32_t r = 0; r < d.nfan; ++r) {
                            const int32_t dev = p->fan[d.fan_off + r];
                            const uint64_t dbytes = uint64_t(p->dst_local_numel[dev] * p->es);
                            const uint64_t q = d.dst_base + uint32_t(at.dst + a * d.ds[0] + j * 16u);
                            if (nv == vpe && ast && q % 16 != 0)
                                return fail(RESHARD_EINVAL, "internal: transpose vector store misaligned");
                            if (q + nv * es > dbytes) return fail(RESHARD_EINVAL, "internal: transpose store outside its destination shard");
                            std::memcpy(static_cast<char *>(dst_ptrs[dev]) + q, y, nv * es);
                        }
                    }
                }
                continue;
            }
            if (di >= p->n_direct + p->n_gather && di < p->n_direct + p->n_gather + p->n_gather_u) {
                // unaligned row-gather chunk: the kernel's slot -> pieces arithmetic
                const uint32_t rb = d.vpr, ns = d.pad[1];
                if (d.pad[0] + ns > p->segs.size() || ns == 0) return fail(RESHARD_EINVAL, "internal: segment table range");
                const rs::Seg *sg = &p->segs[d.pad[0]];
                if (sg[0].col != 0) return fail(RESHARD_EINVAL, "internal: first segment does not start the row");
                auto find_segment = [&](uint32_t col) {
                    uint32_t g = rs::fastdiv(col, d.batch, d.pad[2]);
                    if (g >= ns) g = ns - 1;
                    while (g > 0 && col < sg[g].col) --g;
                    while (g + 1 < ns && col >= sg[g + 1].col) ++g;
                    return g;
                };
                // copy piece [col, col + len) of segment g, row `row`, to out
                auto piece = [&](uint32_t row, uint32_t g, uint32_t col, uint32_t len, uint8_t *out) -> bool {
                    const uint32_t send = g + 1 < ns ? sg[g + 1].col : rb;
                    if (col < sg[g].col || col + len > send) return false;
                    uint32_t i1 = 0, i2 = 0, i3 = 0;
                    if (levels == 1) rs::row_indices<1>(d, row, i1, i2, i3);
                    else if (levels == 2) rs::row_indices<2>(d, row, i1, i2, i3);
                    else rs::row_indices<3>(d, row, i1, i2, i3);
                    const uint32_t off = i1 * sg[g].ss[0] + i2 * sg[g].ss[1] + i3 * sg[g].ss[2] + (col - sg[g].col);
                    const uint64_t q = sg[g].src_base + off;
                    if (q + len > uint64_t(p->src_local_numel[sg[g].buf] * p->es)) return false;
                    std::memcpy(out, static_cast<const char *>(src_ptrs[sg[g].buf]) + q, len);
                    return true;
                };
                if (d.kind & rs::kUnitGather) {
                    // unit gather: the kernel's unit -> (row, segment, offset) arithmetic
                    const uint32_t upr = d.vpr, rbytes = d.run;
                    for (uint32_t v = d.v0; v < d.v1; ++v) {
                        const uint32_t r = rs::fastdiv(v, d.mul_vpr, d.sh_vpr), j = v - r * upr;
                        uint32_t g = rs::fastdiv(j, d.batch, d.pad[2]);
                        if (g >= ns) g = ns - 1;
                        while (g > 0 && j < sg[g].pad) --g;
                        while (g + 1 < ns && j >= sg[g + 1].pad) ++g;
                        const uint32_t w = (g + 1 < ns ? sg[g + 1].col : rbytes) - sg[g].col;
                        if (w < 16 && !(d.ds[0] & rs::kUShortSegs))
                            return fail(RESHARD_EINVAL, "internal: unit gather segment under 16 bytes, unflagged");
                        const uint32_t n = std::min(w, 16u);  // a segment under 16 bytes is one unit
                        const uint32_t o = w < 16 ? 0u : std::min(16u * (j - sg[g].pad), w - 16u);
                        uint8_t out[16];
                        uint32_t i1 = 0, i2 = 0, i3 = 0;
                        if (levels == 1) rs::row_indices<1>(d, d.ss[0] + r, i1, i2, i3);
                        else if (levels == 2) rs::row_indices<2>(d, d.ss[0] + r, i1, i2, i3);
                        else rs::row_indices<3>(d, d.ss[0] + r, i1, i2, i3);
                        const uint64_t q = sg[g].src_base + uint32_t(i1 * sg[g].ss[0] + i2 * sg[g].ss[1] +
                                                                     i3 * sg[g].ss[2] + o);
                        if (o + n > w || q + n > uint64_t(p->src_local_numel[sg[g].buf] * p->es))
                            return fail(RESHARD_EINVAL, "internal: unit gather load outside its segment or shard");
                        std::memcpy(out, static_cast<const char *>(src_ptrs[sg[g].buf]) + q, n);
                        const uint64_t doff = uint64_t((r - d.ss[1]) * rbytes + sg[g].col + o);
                        for (uint32_t q = 0; q < d.nfan; ++q) {
                            const int32_t dev = p->fan[d.fan_off + q];
                            if (d.dst_base + doff + n > uint64_t(p->dst_local_numel[dev] * p->es))
                                return fail(RESHARD_EINVAL, "internal: unit gather store outside its destination shard");
                            std::memcpy(static_cast<char *>(dst_ptrs[dev]) + d.dst_base + doff, out, n);
                        }
                    }
                    continue;
                }
                for (uint32_t ls = d.v0; ls < d.v1; ++ls) {
                    const uint32_t c0 = 16u * ls;
                    const uint32_t lo = std::max(c0, d.ss[2]), hi = std::min(c0 + 16u, d.src_rel0);
                    if (lo >= hi) continue;
                    uint8_t out[16];
                    const uint32_t t = lo + d.ss[1];
                    const uint32_t dr = rs::fastdiv(t, d.mul_vpr, d.sh_vpr);
                    uint32_t row = d.ss[0] + dr, col = t - dr * rb;
                    uint32_t g = find_segment(col);
                    const uint32_t send = g + 1 < ns ? sg[g + 1].col : rb;
                    // pieces in turn: the rest of this segment (or row), then
                    // the next segments (any number when segments are short)
                    uint32_t at = lo, send_g = send;
                    for (;;) {
                        const uint32_t e = at + std::min(hi - at, send_g - col);
                        if (!piece(row, g, col, e - at, out + (at - c0)))
                            return fail(RESHARD_EINVAL, "internal: unaligned gather piece outside its segment or shard");
                        if (e >= hi) break;
                        if (send_g == rb) {
                            ++row;
                            col = 0;
                            g = 0;
                        } else {
                            col = send_g;
                            ++g;
                        }
                        if (g >= ns) return fail(RESHARD_EINVAL, "internal: unaligned gather segment index out of range");
                        send_g = g + 1 < ns ? sg[g + 1].col : rb;
                        at = e;
                    }
                    for (uint32_t r = 0; r < d.nfan; ++r) {
                        const int32_t dev = p->fan[d.fan_off + r];
                        if (d.dst_base + hi > uint64_t(p->dst_local_numel[dev] * p->es))
                            return fail(RESHARD_EINVAL, "internal: unaligned gather store outside its destination shard");
                        std::memcpy(static_cast<char *>(dst_ptrs[dev]) + d.dst_base + lo, out + (lo - c0), hi - lo);
                    }
                }
                continue;
            }
            if (di >= p->n_direct && di < p->n_direct + p->n_gather) {
                // row-gather chunk: the kernel's slot -> (row, segment) arithmetic
                const uint32_t spr = d.vpr, sps = d.run;
                if (d.pad[0] + d.pad[1] > p->segs.size()) return fail(RESHARD_EINVAL, "internal: segment table range");
                for (uint32_t v = d.v0; v < d.v1; ++v) {
                    const uint32_t row = rs::fastdiv(v, d.mul_vpr, d.sh_vpr), j = v - row * spr;
                    const uint32_t g = rs::fastdiv(j, d.batch, d.pad[2]), jj = j - g * sps;
                    if (g >= d.pad[1]) return fail(RESHARD_EINVAL, "internal: segment index out of range");
                    uint32_t i1 = 0, i2 = 0, i3 = 0;
                    if (levels == 1) rs::row_indices<1>(d, row, i1, i2, i3);
                    else if (levels == 2) rs::row_indices<2>(d, row, i1, i2, i3);
                    else rs::row_indices<3>(d, row, i1, i2, i3);
                    const uint32_t dr = i1 * d.ds[0] + i2 * d.ds[1] + i3 * d.ds[2] + 16u * j - d.dst_rel0;
                    const rs::Seg &sg = p->segs[d.pad[0] + g];
                    const uint32_t sr = i1 * sg.ss[0] + i2 * sg.ss[1] + i3 * sg.ss[2] + 16u * jj;
                    if (sg.src_base + sr + 16 > uint64_t(p->src_local_numel[sg.buf] * p->es))
                        return fail(RESHARD_EINVAL, "internal: gather load outside its source shard");
                    const char *src = static_cast<const char *>(src_ptrs[sg.buf]) + sg.src_base + sr;
                    for (uint32_t r = 0; r < d.nfan; ++r) {
                        if (d.dst_base + dr + 16 > uint64_t(p->dst_local_numel[p->fan[d.fan_off + r]] * p->es))
                            return fail(RESHARD_EINVAL, "internal: gather store outside its destination shard");
                        char *dst = static_cast<char *>(dst_ptrs[p->fan[d.fan_off + r]]) + d.dst_base + dr;
                        std::memcpy(dst, src, 16);
                    }
                }
                continue;
            }
            // a source index past the source mesh names a destination buffer
            // (the all-gather strategy's second phase)
            const int64_t sbuf = int64_t(d.src_buf);
            const char *src = static_cast<const char *>(sbuf < p->src.ndev ? src_ptrs[sbuf] : dst_ptrs[sbuf - p->src.ndev]) +
                              d.src_base;
            if (rs::kind_realign(d.kind) && !(p->flags & RESHARD_LDS_STAGING)) {
                // The kernel's shifted-load realignment, same arithmetic: every
                // loaded word must hold a byte of its row.
                const uint32_t m = d.vpr, run = d.run, sb = uint32_t(d.src_base), db = uint32_t(d.dst_base);
                const uint32_t n = (d.v1 - d.v0) * m;
                auto load_word = [&](const rs::Rel &o, uint32_t sph, int32_t j, uint32_t out[4]) -> bool {
                    const int32_t off = int32_t(o.src - sph + 16u * uint32_t(j));
                    const int64_t rel = int64_t(off) - int64_t(o.src);  // row-relative word start
                    if (rel + 16 <= 0 || rel >= int64_t(run)) return false;
                    if (((sb + uint32_t(off)) & 15u) != 0) return false;
                    uint8_t b[16] = {0};
                    for (int64_t t = 0; t < 16; ++t)
                        if (rel + t >= 0 && rel + t < int64_t(run)) b[t] = uint8_t(src[int64_t(off) + t]);
                    std::memcpy(out, b, 16);
                    return true;
                };
                for (uint32_t i = 0; i < n; ++i) {
                    const uint32_t br = rs::fastdiv(i, d.mul_vpr, d.sh_vpr), k = i - br * m;
                    const rs::Rel o = levels == 1 ? rs::row_offsets<1>(d, d.v0 + br)
                                      : levels == 2 ? rs::row_offsets<2>(d, d.v0 + br) : rs::row_offsets<3>(d, d.v0 + br);
                    const uint32_t sph = (sb + o.src) & 15u, tph = (db + o.dst) & 15u;
                    const int32_t start = int32_t(16u * k) - int32_t(tph);
                    const int32_t lo = std::max(start, 0), hi = std::min(start + 16, int32_t(run));
                    if (lo >= hi) continue;
                    const int32_t pos = int32_t(sph) + start;
                    const int32_t j0 = pos >> 4;
                    uint32_t w[8] = {0};
                    if (j0 >= 0 && !load_word(o, sph, j0, w)) return fail(RESHARD_EINVAL, "internal: shifted load outside its row");
                    if (16 * (j0 + 1) < int32_t(sph + run) && !load_word(o, sph, j0 + 1, w + 4))
                        return fail(RESHARD_EINVAL, "internal: shifted load outside its row");
                    const uint32_t sh = uint32_t(pos) & 15u, t4 = sh >> 2, b = sh & 3u;
                    uint32_t v[4];
                    for (uint32_t t = 0; t < 4; ++t) v[t] = rs::align_byte(w[t4 + t + 1], w[t4 + t], b);
                    uint8_t bytes[16];
                    std::memcpy(bytes, v, 16);
                    for (uint32_t r = 0; r < d.nfan; ++r) {
                        char *dst = static_cast<char *>(dst_ptrs[p->fan[d.fan_off + r]]) + d.dst_base + o.dst;
                        for (int32_t c = lo; c < hi; ++c) dst[c] = char(bytes[c - start]);
                    }
                }
                continue;
            }
            if (rs::kind_realign(d.kind)) {
                // Same staging layout, slot arithmetic and dword funnel shifts as
                // the kernel's LDS path, with every staging access bounds-checked.
                const uint32_t m = d.vpr, run = d.run, sb = uint32_t(d.src_base), db = uint32_t(d.dst_base);
                lds.assign(rs::realign_lds_bytes(d.batch, m), 0);
                auto row_off = [&](uint32_t row) {
                    return levels == 1 ? rs::row_offsets<1>(d, row)
                           : levels == 2 ? rs::row_offsets<2>(d, row) : rs::row_offsets<3>(d, row);
                };
                for (uint32_t r0 = d.v0; r0 < d.v1; r0 += d.batch) {
                    const uint32_t nb = std::min(d.batch, d.v1 - r0);
                    std::fill(lds.begin(), lds.end(), 0);
                    for (uint32_t i = 0; i < nb * m; ++i) {
                        const uint32_t br = rs::fastdiv(i, d.mul_vpr, d.sh_vpr), j = i - br * m;
                        const rs::Rel o = row_off(r0 + br);
                        const uint32_t ph = (sb + o.src) & 15u;
                        if (16u * j >= ph + run) continue;
                        const uint32_t at = rs::kRealignFront + 16u * i;
                        if (at + 16u > lds.size()) return fail(RESHARD_EINVAL, "internal: staging write out of range");
                        // the kernel's signed 32-bit word offset; copy only the
                        // row's bytes of the aligned source word
                        const int32_t off = int32_t(o.src + 16u * j - ph);
                        const int64_t wbeg = int64_t(o.src) - ph + 16 * int64_t(j);
                        if (int64_t(off) != wbeg) return fail(RESHARD_EINVAL, "internal: staging word offset wraps");
                        if (((sb + uint32_t(off)) & 15u) != 0) return fail(RESHARD_EINVAL, "internal: staging word misaligned");
                        for (int64_t b = 0; b < 16; ++b) {
                            const int64_t pos = wbeg + b - int64_t(o.src);  // row-relative
                            if (pos >= 0 && pos < int64_t(run)) lds[at + b] = uint8_t(src[wbeg + b]);
                        }
                    }
                    for (uint32_t i = 0; i < nb * m; ++i) {
                        const uint32_t br = rs::fastdiv(i, d.mul_vpr, d.sh_vpr), k = i - br * m;
                        const rs::Rel o = row_off(r0 + br);
                        const uint32_t sph = (sb + o.src) & 15u, tph = (db + o.dst) & 15u;
                        const int32_t start = int32_t(16u * k) - int32_t(tph);
                        const int32_t lo = std::max(start, 0), hi = std::min(start + 16, int32_t(run));
                        if (lo >= hi) continue;
                        const uint32_t q = rs::kRealignFront + br * m * 16u + uint32_t(int32_t(sph) + start);
                        const uint32_t q4 = q >> 2, sh = q & 3u;
                        if (4u * (q4 + 5u) > lds.size()) return fail(RESHARD_EINVAL, "internal: staging read out of range");
                        uint32_t wd[5];
                        std::memcpy(wd, lds.data() + 4u * q4, sizeof(wd));
                        uint32_t v[4];
                        for (int t = 0; t < 4; ++t) v[t] = rs::align_byte(wd[t + 1], wd[t], sh);
                        uint8_t bytes[16];
                        std::memcpy(bytes, v, 16);
                        for (uint32_t r = 0; r < d.nfan; ++r) {
                            char *dst = static_cast<char *>(dst_ptrs[p->fan[d.fan_off + r]]) + d.dst_base + o.dst;
                            for (int32_t b = lo; b < hi; ++b) dst[b] = char(bytes[b - start]);
                        }
                    }
                }
                continue;
            }
            const uint64_t sbytes = uint64_t(
                (sbuf < p->src.ndev ? p->src_local_numel[sbuf] : p->dst_local_numel[sbuf - p->src.ndev]) * p->es);
            for (uint32_t v = d.v0; v < d.v1; ++v) {
                const rs::Rel o = levels == 1   ? rs::chunk_offsets<1>(d, v, w)
                                  : levels == 2 ? rs::chunk_offsets<2>(d, v, w)
                                                : rs::chunk_offsets<3>(d, v, w);
                if (d.src_base + o.src + w > sbytes)
                    return fail(RESHARD_EINVAL, "internal: load outside its source shard");
                for (uint32_t r = 0; r < d.nfan; ++r) {
                    const int32_t dev = p->fan[d.fan_off + r];
                    if (d.dst_base + o.dst + w > uint64_t(p->dst_local_numel[dev] * p->es))
                        return fail(RESHARD_EINVAL, "internal: store outside its destination shard");
                    char *dst = static_cast<char *>(dst_ptrs[dev]) + d.dst_base;
                    std::memcpy(dst + o.dst, src + o.src, w);
                }
            }
        }
        return RESHARD_OK;
    });
}

const char *reshard_last_error(void) { return rs::g_last_error.c_str(); }

const char *reshard_version(void) { return "0.1.0"; }

}  // extern "C"
