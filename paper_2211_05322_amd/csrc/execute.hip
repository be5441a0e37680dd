// execute.hip -- the fused pack / multicast / unpack kernel for gfx950 and
// reshard_execute.
//
// One workgroup runs one descriptor (a chunk of one piece of one unit task).
// Each lane moves W-byte vectors: one load from the sender's buffer, then the
// same vector is stored to every receiver at the same local offset -- the
// broadcast strategy of Section 3.1 (one sender per slice, every receiver
// gets it) with the source read exactly once.  Loads of a batch of U vectors
// are issued before any of their stores so each lane keeps U loads in flight.
// No arithmetic is done on the data, so no MFMA: the kernel is bound by HBM.
//
// Pointer tables travel in the kernel arguments (no per-call upload); the
// descriptor table and receiver lists are read through the constant address
// space so they land in scalar registers.
#include <hip/hip_runtime.h>

#include <string>

#include "../../include/reshard.h"
#include "planner.hpp"

namespace rs {

reshard_status_t fail(reshard_status_t st, const std::string &msg);

#define RS_CONST __attribute__((address_space(4)))

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

template <int W> struct Vec;
template <> struct Vec<16> { typedef u32x4 T; };
template <> struct Vec<8> { typedef u32x2 T; };
template <> struct Vec<4> { typedef unsigned int T; };
template <> struct Vec<2> { typedef unsigned short T; };
template <> struct Vec<1> { typedef unsigned char T; };

template <int NPTR>
struct KArgs {
    const Desc *descs;
    const int32_t *fan;
    uint32_t ndesc;
    uint32_t nsrc;     // ptr[0, nsrc) are source buffers, ptr[nsrc, ...) destination buffers
    uint32_t per_xcd;  // > 0: XCD x runs chunks [x*per_xcd, (x+1)*per_xcd)
    uint32_t pad;
    void *ptr[NPTR];
};

// Build knobs (defaults are the measured best): vectors in flight per lane,
// and the non-temporal hint on source loads / receiver stores.
#ifndef RS_UNROLL
#define RS_UNROLL 4
#endif
#ifndef RS_NT_LOAD
#define RS_NT_LOAD 1
#endif
#ifndef RS_NT_STORE
#define RS_NT_STORE 1
#endif

template <typename V>
__device__ __forceinline__ V load_vec(const V *p) {
    if constexpr (RS_NT_LOAD) return __builtin_nontemporal_load(p);
    else return *p;
}

template <typename V>
__device__ __forceinline__ void store_vec(V *p, V x) {
    if constexpr (RS_NT_STORE) __builtin_nontemporal_store(x, p);
    else *p = x;
}

template <int W, int L, int NPTR>
__device__ __forceinline__ void run_chunk(const Desc &d, const KArgs<NPTR> &a) {
    typedef typename Vec<W>::T V;
    constexpr int U = RS_UNROLL;
    const char *src = static_cast<const char *>(a.ptr[d.src_buf]);
    const RS_CONST int32_t *fan = (const RS_CONST int32_t *)(a.fan + d.fan_off);
    const uint32_t nthr = blockDim.x;
    const uint32_t end = d.v1;
    for (uint32_t v = d.v0 + threadIdx.x; v < end; v += U * nthr) {
        V x[U];
        uint64_t doff[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t vi = v + u * nthr;
            if (vi < end) {
                const Offsets o = piece_offsets<L>(d, vi, W);
                x[u] = load_vec(reinterpret_cast<const V *>(src + o.src));
                doff[u] = o.dst;
            }
        }
        for (uint32_t r = 0; r < d.nfan; ++r) {
            char *dst = static_cast<char *>(a.ptr[a.nsrc + uint32_t(fan[r])]);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t vi = v + u * nthr;
                if (vi < end) store_vec(reinterpret_cast<V *>(dst + doff[u]), x[u]);
            }
        }
    }
}

template <int NPTR>
__global__ __launch_bounds__(1024) void reshard_kernel(KArgs<NPTR> a) {
    const uint32_t b = blockIdx.x;
    const uint32_t idx = a.per_xcd ? (b & 7u) * a.per_xcd + (b >> 3) : b;
    if (idx >= a.ndesc) return;
    // uniform load through the constant address space -> scalar registers
    const RS_CONST u32x4 *q = (const RS_CONST u32x4 *)(a.descs + idx);
    u32x4 raw[sizeof(Desc) / 16];
#pragma unroll
    for (int i = 0; i < int(sizeof(Desc) / 16); ++i) raw[i] = q[i];
    Desc d;
    __builtin_memcpy(&d, raw, sizeof(Desc));
    switch (d.kind) {
        case make_kind(4, 1): run_chunk<16, 1>(d, a); break;
        case make_kind(4, 2): run_chunk<16, 2>(d, a); break;
        case make_kind(4, 3): run_chunk<16, 3>(d, a); break;
        case make_kind(3, 1): run_chunk<8, 1>(d, a); break;
        case make_kind(3, 2): run_chunk<8, 2>(d, a); break;
        case make_kind(3, 3): run_chunk<8, 3>(d, a); break;
        case make_kind(2, 1): run_chunk<4, 1>(d, a); break;
        case make_kind(2, 2): run_chunk<4, 2>(d, a); break;
        case make_kind(2, 3): run_chunk<4, 3>(d, a); break;
        case make_kind(1, 1): run_chunk<2, 1>(d, a); break;
        case make_kind(1, 2): run_chunk<2, 2>(d, a); break;
        case make_kind(1, 3): run_chunk<2, 3>(d, a); break;
        case make_kind(0, 1): run_chunk<1, 1>(d, a); break;
        case make_kind(0, 2): run_chunk<1, 2>(d, a); break;
        case make_kind(0, 3): run_chunk<1, 3>(d, a); break;
        default: break;
    }
}

// ------------------------------------------------------------------ host

namespace {

reshard_status_t hip_fail(const char *what, hipError_t e) {
    return fail(RESHARD_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Upload [descs | fan] to the current device once; returns the device pointer.
reshard_status_t device_table(const Plan &p, int dev, const Desc **descs, const int32_t **fan) {
    if (dev < 0 || dev >= Plan::kMaxHipDevices)
        return fail(RESHARD_EUNSUPPORTED, "HIP device ordinal " + std::to_string(dev) + " above the plan's limit");
    std::lock_guard<std::mutex> lock(p.mu);
    const size_t dbytes = p.descs.size() * sizeof(Desc);
    if (!p.d_table[dev]) {
        const size_t fbytes = p.fan.size() * sizeof(int32_t);
        void *mem = nullptr;
        hipError_t e = hipMalloc(&mem, dbytes + fbytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(RESHARD_ENOMEM, std::string("hipMalloc of the descriptor table: ") + hipGetErrorString(e));
        }
        e = hipMemcpy(mem, p.descs.data(), dbytes, hipMemcpyHostToDevice);
        if (e == hipSuccess && fbytes)
            e = hipMemcpy(static_cast<char *>(mem) + dbytes, p.fan.data(), fbytes, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            (void)hipFree(mem);
            return hip_fail("upload of the descriptor table", e);
        }
        p.d_table[dev] = mem;
    }
    *descs = static_cast<const Desc *>(p.d_table[dev]);
    *fan = reinterpret_cast<const int32_t *>(static_cast<const char *>(p.d_table[dev]) + dbytes);
    return RESHARD_OK;
}

template <int NPTR>
reshard_status_t launch(const Plan &p, const Desc *descs, const int32_t *fan, void *const *src_ptrs,
                        void *const *dst_ptrs, hipStream_t stream) {
    KArgs<NPTR> a;
    a.descs = descs;
    a.fan = fan;
    a.ndesc = uint32_t(p.descs.size());
    a.nsrc = uint32_t(p.src.ndev);
    a.pad = 0;
    for (int64_t k = 0; k < p.src.ndev; ++k) a.ptr[k] = src_ptrs[k];
    for (int64_t k = 0; k < p.dst.ndev; ++k) a.ptr[p.src.ndev + k] = dst_ptrs[k];
    uint32_t grid = a.ndesc;
    a.per_xcd = 0;
    if (!(p.flags & RESHARD_NO_XCD_REMAP)) {
        a.per_xcd = (a.ndesc + 7u) / 8u;
        grid = a.per_xcd * 8u;
    }
    hipLaunchKernelGGL(reshard_kernel<NPTR>, dim3(grid), dim3(uint32_t(p.tuning.block_threads)), 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail("kernel launch", e);
    return RESHARD_OK;
}

}  // namespace

void release_device_table(const Plan &p) {
    std::lock_guard<std::mutex> lock(p.mu);
    int cur = -1;
    bool have_cur = hipGetDevice(&cur) == hipSuccess;
    for (int dev = 0; dev < Plan::kMaxHipDevices; ++dev) {
        if (!p.d_table[dev]) continue;
        if (hipSetDevice(dev) == hipSuccess) (void)hipFree(p.d_table[dev]);
        p.d_table[dev] = nullptr;
    }
    if (have_cur) (void)hipSetDevice(cur);
    (void)hipGetLastError();
}

}  // namespace rs

extern "C" reshard_status_t reshard_execute(const reshard_plan_t *plan, void *const *src_ptrs,
                                            void *const *dst_ptrs, void *stream) {
    using namespace rs;
    const Plan *p = reinterpret_cast<const Plan *>(plan);
    if (!p || !src_ptrs || !dst_ptrs) return fail(RESHARD_EINVAL, "NULL plan or pointer array");
    for (int64_t k = 0; k < p->src.ndev; ++k) {
        if (p->src_local_numel[k] == 0) continue;
        if (!src_ptrs[k])
            return fail(RESHARD_EINVAL, "source buffer " + std::to_string(k) + " is NULL but its shard is not empty");
        if (reinterpret_cast<uintptr_t>(src_ptrs[k]) % uintptr_t(p->align))
            return fail(RESHARD_EINVAL, "source buffer " + std::to_string(k) + " is not aligned to " +
                                            std::to_string(p->align) + " bytes");
    }
    for (int64_t k = 0; k < p->dst.ndev; ++k) {
        if (p->dst_local_numel[k] == 0) continue;
        if (!dst_ptrs[k])
            return fail(RESHARD_EINVAL,
                        "destination buffer " + std::to_string(k) + " is NULL but its shard is not empty");
        if (reinterpret_cast<uintptr_t>(dst_ptrs[k]) % uintptr_t(p->align))
            return fail(RESHARD_EINVAL, "destination buffer " + std::to_string(k) + " is not aligned to " +
                                            std::to_string(p->align) + " bytes");
    }
    if (p->descs.empty()) return RESHARD_OK;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(RESHARD_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    const Desc *descs = nullptr;
    const int32_t *fan = nullptr;
    reshard_status_t st = device_table(*p, dev, &descs, &fan);
    if (st != RESHARD_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (p->src.ndev + p->dst.ndev <= 64) return launch<64>(*p, descs, fan, src_ptrs, dst_ptrs, s);
    return launch<RESHARD_MAX_BUFFERS>(*p, descs, fan, src_ptrs, dst_ptrs, s);
}
