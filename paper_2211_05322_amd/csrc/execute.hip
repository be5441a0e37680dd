// execute.hip -- the resharding kernels for gfx950 and reshard_execute.
//
// Every kernel moves bytes from senders' buffers to receivers' buffers in the
// broadcast strategy of Section 3.1: each unique slice is read once and every
// receiver gets the same bytes at the same local offset.  One workgroup runs
// one descriptor (a chunk); an execute launches one kernel per kind of chunk
// the plan holds:
//   reshard_kernel          direct chunks: a range of W-byte vectors of one
//                           piece of one unit task (source and destination in
//                           the same 16-byte phase);
//   reshard_gather_kernel   row gather: 16-byte slots of whole destination
//                           rows, each from the sender owning its column
//                           segment (equal, 16-byte aligned segments);
//   reshard_gather_u_kernel unaligned row gather: 16-byte slots of the
//                           receivers' buffers built from at most two
//                           misaligned pieces (segments of any width >= 16 B);
//   reshard_realign_kernel  rows in different 16-byte phases, one task at a
//                           time (shifted loads, or staging through LDS).
// Loads of a batch are issued before its stores so each lane keeps several
// loads in flight.  No arithmetic is done on the data, so no MFMA: the
// kernels are bound by HBM.
//
// Pointer tables travel in the kernel arguments (no per-call upload); the
// descriptor table and receiver lists are read through the constant address
// space so they land in scalar registers.
#include <hip/hip_runtime.h>

#include <string>

#include "../../include/reshard.h"
#include "planner.hpp"
#include "status.hpp"

namespace rs {

#define RS_CONST __attribute__((address_space(4)))
#define RS_GLOBAL __attribute__((address_space(1)))

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
    const Seg *segs;   // row-gather segment entries
    uint32_t ndesc;
    uint32_t nsrc;     // ptr[0, nsrc) are source buffers, ptr[nsrc, ...) destination buffers
    uint32_t per_xcd;  // > 0: XCD x runs chunks [x*per_xcd, (x+1)*per_xcd)
    uint32_t pad;
    void *ptr[NPTR];
};

// Build knobs (defaults are the measured best): vectors in flight per lane,
// and the non-temporal hint on source loads / receiver stores.
#ifndef RS_UNROLL
#define RS_UNROLL 2
#endif
#ifndef RS_NT_LOAD
#define RS_NT_LOAD 0
#endif
#ifndef RS_NT_STORE
#define RS_NT_STORE 1
#endif

template <typename V>
__device__ __forceinline__ V load_vec(const RS_GLOBAL V *p) {
    if constexpr (RS_NT_LOAD) return __builtin_nontemporal_load(p);
    else return *p;
}

template <typename V>
__device__ __forceinline__ void store_vec(RS_GLOBAL V *p, V x) {
    if constexpr (RS_NT_STORE) __builtin_nontemporal_store(x, p);
    else *p = x;
}

#ifndef RS_PIPELINE
#define RS_PIPELINE 1
#endif
#ifndef RS_DRAIN
#define RS_DRAIN 0  // 1: wait for a batch's stores before the next batch's loads
#endif
#ifndef RS_STORE_ORDER
#define RS_STORE_ORDER 0  // 0: receiver-major stores, 1: vector-major stores
#endif

// Descriptor idx, loaded with a uniform index through the constant address
// space so it lands in scalar registers.
template <int NPTR>
__device__ __forceinline__ Desc load_desc(const RS_CONST KArgs<NPTR> *a, uint32_t idx) {
    const RS_CONST u32x4 *q = (const RS_CONST u32x4 *)(a->descs + idx);
    u32x4 raw[sizeof(Desc) / 16];
#pragma unroll
    for (int i = 0; i < int(sizeof(Desc) / 16); ++i) raw[i] = q[i];
    Desc d;
    __builtin_memcpy(&d, raw, sizeof(Desc));
    return d;
}

// Load one batch of U vectors per lane (vectors v, v+nthr, ...).  FULL: the
// whole batch is inside the chunk (a workgroup-uniform fact), so no lane
// needs a bounds check and the loop carries no divergent branches.
template <int W, int L, int U, bool FULL>
__device__ __forceinline__ void load_batch(const Desc &d, const RS_GLOBAL char *src, uint32_t v, uint32_t nthr,
                                           uint32_t end, typename Vec<W>::T (&x)[U], uint32_t (&doff)[U]) {
    typedef typename Vec<W>::T V;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint32_t vi = v + u * nthr;
        if (FULL || vi < end) {
            const Rel o = chunk_offsets<L>(d, vi, W);
            x[u] = load_vec((const RS_GLOBAL V *)(src + o.src));
            doff[u] = o.dst;
        }
    }
}

// Store one batch to every receiver.  RF > 0: the fan-out is a compile-time
// constant (straight-line stores, so the wait counts stay exact); RF == 0:
// runtime receiver count.  ORDER 0: receiver-major, 1: vector-major (every
// receiver's copy of one vector before the next vector; compile-time fan-out
// only).
template <int W, int U, int RF, bool FULL, int ORDER = RS_STORE_ORDER, int NPTR>
__device__ __forceinline__ void store_batch(const Desc &d, const RS_CONST KArgs<NPTR> *a, const RS_CONST int32_t *fan,
                                            uint32_t v, uint32_t nthr, uint32_t end,
                                            const typename Vec<W>::T (&x)[U], const uint32_t (&doff)[U]) {
    typedef typename Vec<W>::T V;
    const uint32_t nr = RF > 0 ? uint32_t(RF) : d.nfan;
    if (ORDER == 1 && RF > 0) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t vi = v + u * nthr;
#pragma unroll
            for (uint32_t r = 0; r < nr; ++r) {
                RS_GLOBAL char *dst = (RS_GLOBAL char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base;
                if (FULL || vi < end) store_vec((RS_GLOBAL V *)(dst + doff[u]), x[u]);
            }
        }
    } else {
#pragma unroll
        for (uint32_t r = 0; r < nr; ++r) {
            RS_GLOBAL char *dst = (RS_GLOBAL char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t vi = v + u * nthr;
                if (FULL || vi < end) store_vec((RS_GLOBAL V *)(dst + doff[u]), x[u]);
            }
        }
    }
    if (RS_DRAIN) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

template <int W, int L, int RF, int NPTR>
__device__ __forceinline__ void run_chunk(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    typedef typename Vec<W>::T V;
    constexpr int U = RS_UNROLL;
    const RS_GLOBAL char *src = (const RS_GLOBAL char *)a->ptr[d.src_buf] + d.src_base;
    const RS_CONST int32_t *fan = (const RS_CONST int32_t *)(a->fan + d.fan_off);
    const uint32_t nthr = blockDim.x;
    const uint32_t end = d.v1;
    const uint32_t step = U * nthr;
    const uint32_t tid = threadIdx.x;
    uint32_t base = d.v0;  // workgroup-uniform batch start
    if (RS_PIPELINE) {
        // two register sets: the next batch's loads are in flight while the
        // current batch is stored
        V x[U], y[U];
        uint32_t dx[U], dy[U];
        if (base + step <= end) {
            load_batch<W, L, U, true>(d, src, base + tid, nthr, end, x, dx);
            for (;;) {
                if (base + 2 * step > end) {
                    store_batch<W, U, RF, true>(d, a, fan, base + tid, nthr, end, x, dx);
                    base += step;
                    break;
                }
                load_batch<W, L, U, true>(d, src, base + step + tid, nthr, end, y, dy);
                store_batch<W, U, RF, true>(d, a, fan, base + tid, nthr, end, x, dx);
                base += step;
                if (base + 2 * step > end) {
                    store_batch<W, U, RF, true>(d, a, fan, base + tid, nthr, end, y, dy);
                    base += step;
                    break;
                }
                load_batch<W, L, U, true>(d, src, base + step + tid, nthr, end, x, dx);
                store_batch<W, U, RF, true>(d, a, fan, base + tid, nthr, end, y, dy);
                base += step;
            }
        }
    } else {
        for (; base + step <= end; base += step) {
            V x[U];
            uint32_t doff[U];
            load_batch<W, L, U, true>(d, src, base + tid, nthr, end, x, doff);
            store_batch<W, U, RF, true>(d, a, fan, base + tid, nthr, end, x, doff);
        }
    }
    if (base < end) {  // ragged tail: per-lane bounds checks
        V x[U];
        uint32_t doff[U];
        load_batch<W, L, U, false>(d, src, base + tid, nthr, end, x, doff);
        store_batch<W, U, RF, false>(d, a, fan, base + tid, nthr, end, x, doff);
    }
}

// Write bytes [lo, hi) (0 <= lo < hi <= 16) of the 16-byte value v to
// slot[lo, hi), where slot is 16-byte aligned: naturally aligned 8/4/2/1-byte
// pieces, at most six stores.
__device__ __forceinline__ void store_partial(RS_GLOBAL unsigned char *slot, u32x4 v, uint32_t lo, uint32_t hi) {
    const uint64_t q0 = (uint64_t(v.y) << 32) | v.x, q1 = (uint64_t(v.w) << 32) | v.z;
#pragma nounroll
    while (lo < hi) {
        const uint64_t q = lo < 8 ? q0 : q1;
        const uint32_t sh = 8u * (lo & 7u);
        if ((lo & 7u) == 0 && lo + 8 <= hi) {
            *(RS_GLOBAL uint64_t *)(slot + lo) = q;
            lo += 8;
        } else if ((lo & 3u) == 0 && lo + 4 <= hi) {
            *(RS_GLOBAL uint32_t *)(slot + lo) = uint32_t(q >> sh);
            lo += 4;
        } else if ((lo & 1u) == 0 && lo + 2 <= hi) {
            *(RS_GLOBAL uint16_t *)(slot + lo) = uint16_t(q >> sh);
            lo += 2;
        } else {
            slot[lo] = (unsigned char)(q >> sh);
            lo += 1;
        }
    }
}

// LDS realignment path for rows whose source and destination 16-byte phases
// differ.  Per pass over `batch` rows: (1) every source word a row touches is
// loaded once, 16-byte aligned and coalesced, into the row's staging slot in
// LDS; (2) each lane builds one 16-byte destination slot from five staged
// dwords (v_alignbyte funnel shift by the row's phase difference) and stores
// it, aligned, to every receiver; slots cut by the row's ends are written
// byte by byte.  A source word is loaded only if it holds a byte of the row,
// so it never leaves the row's 4 KiB page.
template <int L, int NPTR>
__device__ __forceinline__ void run_realign(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char rs_lds[];
    const uint32_t m = d.vpr, run = d.run;
    const uint32_t sb = uint32_t(d.src_base), db = uint32_t(d.dst_base);
    const RS_GLOBAL char *src = (const RS_GLOBAL char *)a->ptr[d.src_buf] + d.src_base;
    const RS_CONST int32_t *fan = (const RS_CONST int32_t *)(a->fan + d.fan_off);
    const uint32_t nthr = blockDim.x, tid = threadIdx.x;
    for (uint32_t r0 = d.v0; r0 < d.v1; r0 += d.batch) {
        const uint32_t n = (d.v1 - r0 < d.batch ? d.v1 - r0 : d.batch) * m;
        // stage: up to 4 words per lane per round, all loads issued first
        for (uint32_t i0 = 0; i0 < n; i0 += 4u * nthr) {
            u32x4 w[4];
            bool ok[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint32_t i = i0 + tid + uint32_t(u) * nthr;
                ok[u] = false;
                if (i < n) {
                    const uint32_t br = fastdiv(i, d.mul_vpr, d.sh_vpr);
                    const uint32_t j = i - br * m;
                    const Rel o = row_offsets<L>(d, r0 + br);
                    const uint32_t ph = (sb + o.src) & 15u;
                    if (16u * j < ph + run) {
                        // the word holding the row's first byte can start up to
                        // 15 bytes before the chunk base: a signed offset (chunk
                        // spans stay below 2^31 on this path)
                        const int32_t off = int32_t(o.src + 16u * j - ph);
                        w[u] = load_vec((const RS_GLOBAL u32x4 *)(src + off));
                        ok[u] = true;
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint32_t i = i0 + tid + uint32_t(u) * nthr;
                if (ok[u]) *reinterpret_cast<u32x4 *>(rs_lds + kRealignFront + 16u * i) = w[u];
            }
        }
        __syncthreads();
        for (uint32_t i = tid; i < n; i += nthr) {
            const uint32_t br = fastdiv(i, d.mul_vpr, d.sh_vpr);
            const uint32_t k = i - br * m;
            const Rel o = row_offsets<L>(d, r0 + br);
            const uint32_t sph = (sb + o.src) & 15u, tph = (db + o.dst) & 15u;
            const int32_t start = int32_t(16u * k) - int32_t(tph);  // row-relative slot start
            const int32_t lo = start > 0 ? start : 0;
            const int32_t hi = start + 16 < int32_t(run) ? start + 16 : int32_t(run);
            if (lo >= hi) continue;
            const uint32_t q = kRealignFront + br * m * 16u + uint32_t(int32_t(sph) + start);
            const uint32_t *w = reinterpret_cast<const uint32_t *>(rs_lds) + (q >> 2);
            const uint32_t sh = q & 3u;
            const uint32_t w0 = w[0], w1 = w[1], w2 = w[2], w3 = w[3], w4 = w[4];
            u32x4 v;
            v.x = __builtin_amdgcn_alignbyte(w1, w0, sh);
            v.y = __builtin_amdgcn_alignbyte(w2, w1, sh);
            v.z = __builtin_amdgcn_alignbyte(w3, w2, sh);
            v.w = __builtin_amdgcn_alignbyte(w4, w3, sh);
            if (lo == start && hi == start + 16) {
                for (uint32_t r = 0; r < d.nfan; ++r) {
                    RS_GLOBAL char *dst = (RS_GLOBAL char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base;
                    store_vec((RS_GLOBAL u32x4 *)(dst + (o.dst + uint32_t(start))), v);
                }
            } else {
                for (uint32_t r = 0; r < d.nfan; ++r) {
                    RS_GLOBAL unsigned char *slot =
                        (RS_GLOBAL unsigned char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base + o.dst + start;
                    store_partial(slot, v, uint32_t(lo - start), uint32_t(hi - start));
                }
            }
        }
        __syncthreads();
    }
}

// 16-byte path: fan-outs 1..8 get their own straight-line store sequence.
template <int L, int NPTR>
__device__ __forceinline__ void run_wide(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    switch (d.nfan) {
        case 1: run_chunk<16, L, 1>(d, a); break;
        case 2: run_chunk<16, L, 2>(d, a); break;
        case 3: run_chunk<16, L, 3>(d, a); break;
        case 4: run_chunk<16, L, 4>(d, a); break;
        case 5: run_chunk<16, L, 5>(d, a); break;
        case 6: run_chunk<16, L, 6>(d, a); break;
        case 7: run_chunk<16, L, 7>(d, a); break;
        case 8: run_chunk<16, L, 8>(d, a); break;
        default: run_chunk<16, L, 0>(d, a); break;
    }
}

template <int NPTR>
__global__ __launch_bounds__(1024) void reshard_kernel(KArgs<NPTR> args) {
    // The argument block is read in place through the kernarg segment pointer
    // (constant address space): pointer-table lookups with a uniform index
    // become scalar loads and nothing is copied to private memory.
    const RS_CONST KArgs<NPTR> *a = (const RS_CONST KArgs<NPTR> *)__builtin_amdgcn_kernarg_segment_ptr();
    const uint32_t b = blockIdx.x;
    const uint32_t idx = a->per_xcd ? (b & 7u) * a->per_xcd + (b >> 3) : b;
    if (idx >= a->ndesc) return;
    const Desc d = load_desc(a, idx);
    switch (d.kind) {
        case make_kind(4, 1): run_wide<1>(d, a); break;
        case make_kind(4, 2): run_wide<2>(d, a); break;
        case make_kind(4, 3): run_wide<3>(d, a); break;
        case make_kind(3, 1): run_chunk<8, 1, 0>(d, a); break;
        case make_kind(3, 2): run_chunk<8, 2, 0>(d, a); break;
        case make_kind(3, 3): run_chunk<8, 3, 0>(d, a); break;
        case make_kind(2, 1): run_chunk<4, 1, 0>(d, a); break;
        case make_kind(2, 2): run_chunk<4, 2, 0>(d, a); break;
        case make_kind(2, 3): run_chunk<4, 3, 0>(d, a); break;
        case make_kind(1, 1): run_chunk<2, 1, 0>(d, a); break;
        case make_kind(1, 2): run_chunk<2, 2, 0>(d, a); break;
        case make_kind(1, 3): run_chunk<2, 3, 0>(d, a); break;
        case make_kind(0, 1): run_chunk<1, 1, 0>(d, a); break;
        case make_kind(0, 2): run_chunk<1, 2, 0>(d, a); break;
        case make_kind(0, 3): run_chunk<1, 3, 0>(d, a); break;
        default: break;
    }
}

// Bytes [s, s+16) of the 32-byte value lo:hi (s in 0..15), as four dwords.
__device__ __forceinline__ u32x4 funnel32(u32x4 lo, u32x4 hi, uint32_t s) {
    const uint32_t t = s >> 2, b = s & 3u;
    const uint32_t d0 = lo.x, d1 = lo.y, d2 = lo.z, d3 = lo.w, d4 = hi.x, d5 = hi.y, d6 = hi.z, d7 = hi.w;
    const uint32_t e0 = t == 0 ? d0 : t == 1 ? d1 : t == 2 ? d2 : d3;
    const uint32_t e1 = t == 0 ? d1 : t == 1 ? d2 : t == 2 ? d3 : d4;
    const uint32_t e2 = t == 0 ? d2 : t == 1 ? d3 : t == 2 ? d4 : d5;
    const uint32_t e3 = t == 0 ? d3 : t == 1 ? d4 : t == 2 ? d5 : d6;
    const uint32_t e4 = t == 0 ? d4 : t == 1 ? d5 : t == 2 ? d6 : d7;
    u32x4 v;
    v.x = __builtin_amdgcn_alignbyte(e1, e0, b);
    v.y = __builtin_amdgcn_alignbyte(e2, e1, b);
    v.z = __builtin_amdgcn_alignbyte(e3, e2, b);
    v.w = __builtin_amdgcn_alignbyte(e4, e3, b);
    return v;
}

// Realignment without staging: each lane builds a 16-byte destination slot
// from the two aligned source words that cover it, loaded directly (the
// neighbouring lane's overlapping load is served by the cache), funnel-shifted
// in registers.  Same descriptors as the staging path: slot (row, k) for k <
// m.  Words holding no byte of the row are not loaded.
template <int L, int NPTR>
__device__ __forceinline__ void run_shift(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    constexpr int U = 2;
    const uint32_t m = d.vpr, run = d.run;
    const uint32_t sb = uint32_t(d.src_base), db = uint32_t(d.dst_base);
    const RS_GLOBAL char *src = (const RS_GLOBAL char *)a->ptr[d.src_buf] + d.src_base;
    const RS_CONST int32_t *fan = (const RS_CONST int32_t *)(a->fan + d.fan_off);
    const uint32_t nthr = blockDim.x, tid = threadIdx.x;
    const uint32_t n = (d.v1 - d.v0) * m;
    for (uint32_t i0 = 0; i0 < n; i0 += U * nthr) {
        u32x4 v[U];
        int32_t lo[U], hi[U], st[U];
        uint32_t dof[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t i = i0 + tid + uint32_t(u) * nthr;
            lo[u] = 0;
            hi[u] = 0;
            st[u] = 0;
            dof[u] = 0;
            if (i < n) {
                const uint32_t br = fastdiv(i, d.mul_vpr, d.sh_vpr);
                const uint32_t k = i - br * m;
                const Rel o = row_offsets<L>(d, d.v0 + br);
                const uint32_t sph = (sb + o.src) & 15u, tph = (db + o.dst) & 15u;
                const int32_t start = int32_t(16u * k) - int32_t(tph);
                lo[u] = start > 0 ? start : 0;
                hi[u] = start + 16 < int32_t(run) ? start + 16 : int32_t(run);
                st[u] = start;
                dof[u] = o.dst;
                if (lo[u] < hi[u]) {
                    const int32_t pos = int32_t(sph) + start;  // in the row's word grid, >= -15
                    const int32_t j0 = pos >> 4;                // arithmetic shift: -1 for the head
                    u32x4 w0 = {0u, 0u, 0u, 0u}, w1 = {0u, 0u, 0u, 0u};
                    if (j0 >= 0)
                        w0 = load_vec((const RS_GLOBAL u32x4 *)(src + int32_t(o.src - sph + 16u * uint32_t(j0))));
                    if (16 * (j0 + 1) < int32_t(sph + run))
                        w1 = load_vec((const RS_GLOBAL u32x4 *)(src + int32_t(o.src - sph + 16u * uint32_t(j0 + 1))));
                    v[u] = funnel32(w0, w1, uint32_t(pos) & 15u);
                }
            }
        }
        for (uint32_t r = 0; r < d.nfan; ++r) {
            RS_GLOBAL char *dst = (RS_GLOBAL char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (lo[u] >= hi[u]) continue;
                if (lo[u] == st[u] && hi[u] == st[u] + 16) {
                    store_vec((RS_GLOBAL u32x4 *)(dst + (dof[u] + uint32_t(st[u]))), v[u]);
                } else {
                    RS_GLOBAL unsigned char *slot = (RS_GLOBAL unsigned char *)dst + dof[u] + st[u];
                    store_partial(slot, v[u], uint32_t(lo[u] - st[u]), uint32_t(hi[u] - st[u]));
                }
            }
        }
    }
}

// Row-gather path (see desc.h): a workgroup writes whole destination rows,
// each 16-byte slot loaded from the sender owning its column segment.  The
// chunk's segment entries are staged in LDS once (64-bit source pointer +
// three strides each), then each lane gathers its slots with per-lane
// pointers; stores are the direct path's (receiver bases in scalar
// registers, one shared 32-bit offset).
template <int L, int U, bool FULL>
__device__ __forceinline__ void gather_batch(const Desc &d, const uint64_t *sp, const uint32_t *sst, uint32_t v,
                                             uint32_t nthr, uint32_t end, u32x4 (&x)[U], uint32_t (&doff)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint32_t vi = v + u * nthr;
        if (FULL || vi < end) {
            const uint32_t row = fastdiv(vi, d.mul_vpr, d.sh_vpr);
            const uint32_t j = vi - row * d.vpr;
            const uint32_t g = fastdiv(j, d.batch, d.pad[2]);
            const uint32_t jj = j - g * d.run;
            uint32_t i1, i2, i3;
            row_indices<L>(d, row, i1, i2, i3);
            doff[u] = i1 * d.ds[0] + i2 * d.ds[1] + i3 * d.ds[2] + 16u * j - d.dst_rel0;
            const uint32_t so = i1 * sst[3 * g] + i2 * sst[3 * g + 1] + i3 * sst[3 * g + 2] + 16u * jj;
            x[u] = load_vec((const RS_GLOBAL u32x4 *)(sp[g] + so));
        }
    }
}

extern __shared__ __attribute__((aligned(16))) unsigned char rs_lds[];

// Stage chunk d's segment entries in LDS: 64-bit source pointers at 0,
// three 32-bit strides each at 8 * kMaxSegs.  The caller synchronizes.
template <int NPTR>
__device__ __forceinline__ void stage_segments(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    uint64_t *sp = reinterpret_cast<uint64_t *>(rs_lds);
    uint32_t *sst = reinterpret_cast<uint32_t *>(rs_lds + 8u * kMaxSegs);
    const RS_CONST Seg *segs = (const RS_CONST Seg *)(a->segs + d.pad[0]);
    for (uint32_t g = threadIdx.x; g < d.pad[1]; g += blockDim.x) {
        sp[g] = uint64_t(a->ptr[segs[g].buf]) + segs[g].src_base;
        sst[3 * g] = segs[g].ss[0];
        sst[3 * g + 1] = segs[g].ss[1];
        sst[3 * g + 2] = segs[g].ss[2];
    }
}

template <int L, int RF, int NPTR>
__device__ __forceinline__ void run_gather(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    constexpr int U = RS_UNROLL;
    const uint64_t *sp = reinterpret_cast<const uint64_t *>(rs_lds);
    const uint32_t *sst = reinterpret_cast<const uint32_t *>(rs_lds + 8u * kMaxSegs);
    const uint32_t nthr = blockDim.x, tid = threadIdx.x;
    const RS_CONST int32_t *fan = (const RS_CONST int32_t *)(a->fan + d.fan_off);
    // Store order measured per fan-out: vector-major up to 4 receivers
    // (2 % faster at 4), receiver-major above (1 % faster at 8).
    constexpr int O = RF >= 1 && RF <= 4 ? 1 : 0;
    const uint32_t end = d.v1, step = U * nthr;
    uint32_t base = d.v0;
    u32x4 x[U], y[U];
    uint32_t dx[U], dy[U];
    if (base + step <= end) {
        gather_batch<L, U, true>(d, sp, sst, base + tid, nthr, end, x, dx);
        for (;;) {
            if (base + 2 * step > end) {
                store_batch<16, U, RF, true, O>(d, a, fan, base + tid, nthr, end, x, dx);
                base += step;
                break;
            }
            gather_batch<L, U, true>(d, sp, sst, base + step + tid, nthr, end, y, dy);
            store_batch<16, U, RF, true, O>(d, a, fan, base + tid, nthr, end, x, dx);
            base += step;
            if (base + 2 * step > end) {
                store_batch<16, U, RF, true, O>(d, a, fan, base + tid, nthr, end, y, dy);
                base += step;
                break;
            }
            gather_batch<L, U, true>(d, sp, sst, base + step + tid, nthr, end, x, dx);
            store_batch<16, U, RF, true, O>(d, a, fan, base + tid, nthr, end, y, dy);
            base += step;
        }
    }
    if (base < end) {
        gather_batch<L, U, false>(d, sp, sst, base + tid, nthr, end, x, dx);
        store_batch<16, U, RF, false, O>(d, a, fan, base + tid, nthr, end, x, dx);
    }
}

template <int L, int NPTR>
__device__ __forceinline__ void run_gather_fan(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    switch (d.nfan) {
        case 1: run_gather<L, 1>(d, a); break;
        case 2: run_gather<L, 2>(d, a); break;
        case 3: run_gather<L, 3>(d, a); break;
        case 4: run_gather<L, 4>(d, a); break;
        case 5: run_gather<L, 5>(d, a); break;
        case 6: run_gather<L, 6>(d, a); break;
        case 7: run_gather<L, 7>(d, a); break;
        case 8: run_gather<L, 8>(d, a); break;
        default: run_gather<L, 0>(d, a); break;
    }
}

template <int NPTR>
__device__ __forceinline__ void run_gather_levels(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    switch (kind_levels(d.kind)) {
        case 1: run_gather_fan<1>(d, a); break;
        case 2: run_gather_fan<2>(d, a); break;
        default: run_gather_fan<3>(d, a); break;
    }
}

template <int NPTR>
__global__ __launch_bounds__(1024) void reshard_gather_kernel(KArgs<NPTR> args) {
    const RS_CONST KArgs<NPTR> *a = (const RS_CONST KArgs<NPTR> *)__builtin_amdgcn_kernarg_segment_ptr();
    const uint32_t b = blockIdx.x;
    const uint32_t idx = a->per_xcd ? (b & 7u) * a->per_xcd + (b >> 3) : b;
    if (idx >= a->ndesc) return;
    const Desc d = load_desc(a, idx);
    stage_segments(d, a);
    __syncthreads();
    run_gather_levels(d, a);
}

// Unaligned row gather (see desc.h): a workgroup writes 16-byte slots of the
// receivers' buffers; each slot holds at most two pieces (end of a segment or
// row, start of the next), each read as the aligned source word(s) holding
// it and funnel-shifted into place.  A word is loaded only if it holds a
// byte of its piece, so no load leaves the 4 KiB page of a byte it needs.
// LDS: 64-bit source pointers at 0, three strides per segment at
// 8 * kMaxSegs, segment starts (bytes within the row) at 20 * kMaxSegs.
constexpr uint32_t kGatherULds = 24u * kMaxSegs;
// the same + first units at 24 * kMaxSegs, the short segments' indices at
// 28 * kMaxSegs and their count at 32 * kMaxSegs
constexpr uint32_t kUnitLds = 32u * kMaxSegs + 16u;

// Chunk order of the unaligned row gather: the dispatcher hands workgroups to
// the 8 XCDs in turn, so blocks b, b + 8, ..., b + 8 (kUGroup - 1) share an
// XCD and its L2; they take kUGroup consecutive chunks.  A sender row that
// ends inside a cache line shares it with the sender's next row, which the
// next chunk or the one after gathers: on one XCD that line is fetched once
// (measured reads 1.09 x the unique bytes with round-robin chunks, 1.02 x in
// runs of 16, same time), while the resident chunks still form one window
// of the destination.  The grid is rounded up to whole runs of 8 kUGroup.
constexpr uint32_t kUGroup = 16;

__device__ __forceinline__ uint32_t grouped_chunk(uint32_t b) {
    return (b / (8u * kUGroup)) * (8u * kUGroup) + (b & 7u) * kUGroup + (b >> 3) % kUGroup;
}

template <int NPTR, bool UNITS = false>
__device__ __forceinline__ void stage_segments_u(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    uint64_t *sp = reinterpret_cast<uint64_t *>(rs_lds);
    uint32_t *sst = reinterpret_cast<uint32_t *>(rs_lds + 8u * kMaxSegs);
    uint32_t *scol = reinterpret_cast<uint32_t *>(rs_lds + 20u * kMaxSegs);
    const RS_CONST Seg *segs = (const RS_CONST Seg *)(a->segs + d.pad[0]);
    for (uint32_t g = threadIdx.x; g < d.pad[1]; g += blockDim.x) {
        sp[g] = uint64_t(a->ptr[segs[g].buf]) + segs[g].src_base;
        sst[3 * g] = segs[g].ss[0];
        sst[3 * g + 1] = segs[g].ss[1];
        sst[3 * g + 2] = segs[g].ss[2];
        scol[g] = segs[g].col;
        if (UNITS) {
            reinterpret_cast<uint32_t *>(rs_lds + 24u * kMaxSegs)[g] = segs[g].pad;
            // segments under 16 bytes, listed in any order (the count was
            // cleared before the barrier that precedes this staging)
            if ((d.ds[0] & kUShortSegs) && (g + 1 < d.pad[1] ? segs[g + 1].col : d.run) - segs[g].col < 16u) {
                const uint32_t k = atomicAdd(reinterpret_cast<uint32_t *>(rs_lds + 32u * kMaxSegs), 1u);
                reinterpret_cast<uint32_t *>(rs_lds + 28u * kMaxSegs)[k] = g;
            }
        }
    }
}

// Segment holding row byte `col`: a guess from the nominal width, then the
// staged segment starts decide.
__device__ __forceinline__ uint32_t find_segment(const Desc &d, const uint32_t *scol, uint32_t col) {
    const uint32_t ns = d.pad[1];
    uint32_t g = fastdiv(col, d.batch, d.pad[2]);
    if (g >= ns) g = ns - 1;
    while (g > 0 && col < scol[g]) --g;
    while (g + 1 < ns && col >= scol[g + 1]) ++g;
    return g;
}

template <int L>
__device__ __forceinline__ uint64_t segment_addr(const Desc &d, const uint64_t *sp, const uint32_t *sst,
                                                 const uint32_t *scol, uint32_t g, uint32_t row, uint32_t col) {
    uint32_t i1, i2, i3;
    row_indices<L>(d, row, i1, i2, i3);
    const uint32_t off = i1 * sst[3 * g] + i2 * sst[3 * g + 1] + i3 * sst[3 * g + 2] + (col - scol[g]);
    return sp[g] + off;
}

struct USlot {
    u32x4 a0, a1, b0, b1;   // aligned source words of the two pieces
    uint32_t lo, hi, e1;    // slot bytes [lo, hi) in chunk coordinates; piece 2 starts at e1
    uint32_t sha, shb;      // byte offsets of the pieces in their first words
    uint32_t e2;            // piece 2 ends at e2: hi, unless a segment shorter than the rest follows
    uint32_t row, col, g;   // where the bytes from e2 on start (segments shorter than 16 bytes)
};

template <int L, bool SHORT>
__device__ __forceinline__ void uslot_load(const Desc &d, const uint64_t *sp, const uint32_t *sst,
                                           const uint32_t *scol, uint32_t c0, USlot &s) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    s.a1 = z;
    s.b1 = z;
    s.lo = c0 > d.ss[2] ? c0 : d.ss[2];
    s.hi = c0 + 16u < d.src_rel0 ? c0 + 16u : d.src_rel0;
    s.e1 = s.hi;
    s.e2 = s.hi;
    s.sha = 0;
    s.shb = 0;
    s.row = 0;
    s.col = 0;
    s.g = 0;
    if (s.lo >= s.hi) return;
    const uint32_t rb = d.vpr, ns = d.pad[1];
    const uint32_t t = s.lo + d.ss[1];  // >= 0: the region starts at ss[2] = -cofs0 in the first chunk
    const uint32_t dr = fastdiv(t, d.mul_vpr, d.sh_vpr);
    uint32_t row = d.ss[0] + dr, col = t - dr * rb;
    uint32_t g = find_segment(d, scol, col);
    const uint32_t send = g + 1 < ns ? scol[g + 1] : rb;
    s.e1 = s.lo + ((s.hi - s.lo) < (send - col) ? (s.hi - s.lo) : (send - col));
    uint64_t q = segment_addr<L>(d, sp, sst, scol, g, row, col);
    s.sha = uint32_t(q) & 15u;
    s.a0 = load_vec((const RS_GLOBAL u32x4 *)(q & ~uint64_t(15)));
    if (s.sha + (s.e1 - s.lo) > 16u) s.a1 = load_vec((const RS_GLOBAL u32x4 *)((q & ~uint64_t(15)) + 16u));
    if (s.e1 < s.hi) {
        if (send == rb) {  // the next row's first segment
            ++row;
            col = 0;
            g = 0;
        } else {
            col = send;
            ++g;
        }
        uint32_t send2 = rb;
        if (SHORT) {  // piece 2 may end before the slot does
            send2 = g + 1 < ns ? scol[g + 1] : rb;
            s.e2 = s.e1 + ((s.hi - s.e1) < (send2 - col) ? (s.hi - s.e1) : (send2 - col));
        }
        q = segment_addr<L>(d, sp, sst, scol, g, row, col);
        s.shb = uint32_t(q) & 15u;
        s.b0 = load_vec((const RS_GLOBAL u32x4 *)(q & ~uint64_t(15)));
        if (s.shb + (s.e2 - s.e1) > 16u) s.b1 = load_vec((const RS_GLOBAL u32x4 *)((q & ~uint64_t(15)) + 16u));
        if (SHORT && s.e2 < s.hi) {  // a short segment: the bytes from e2 on come from the pieces after it
            if (send2 == rb) {
                ++row;
                col = 0;
                g = 0;
            } else {
                col = send2;
                ++g;
            }
            s.row = row;
            s.col = col;
            s.g = g;
        }
    }
}

// Slot bytes [e2, hi) of a slot cut by segments shorter than 16 bytes (the
// rare third and later pieces): one byte load each, the segment walk
// continued from (row, col, g).
template <int L>
__device__ __forceinline__ u32x4 uslot_rest(const Desc &d, const uint64_t *sp, const uint32_t *sst,
                                            const uint32_t *scol, const USlot &s, uint32_t c0, u32x4 out) {
    const uint32_t rb = d.vpr, ns = d.pad[1];
    uint32_t row = s.row, col = s.col, g = s.g;
    uint32_t send = g + 1 < ns ? scol[g + 1] : rb;
    uint64_t q = segment_addr<L>(d, sp, sst, scol, g, row, col);
    uint32_t w0 = out.x, w1 = out.y, w2 = out.z, w3 = out.w;
    for (uint32_t k = s.e2 - c0; k < s.hi - c0; ++k) {
        if (col == send) {
            if (send == rb) {
                ++row;
                col = 0;
                g = 0;
            } else {
                ++g;
            }
            send = g + 1 < ns ? scol[g + 1] : rb;
            q = segment_addr<L>(d, sp, sst, scol, g, row, col);
        }
        const uint32_t b = *(const RS_GLOBAL unsigned char *)q;
        const uint32_t sh = 8u * (k & 3u), m = ~(0xFFu << sh);
        const uint32_t wi = k >> 2;
        w0 = wi == 0 ? (w0 & m) | (b << sh) : w0;
        w1 = wi == 1 ? (w1 & m) | (b << sh) : w1;
        w2 = wi == 2 ? (w2 & m) | (b << sh) : w2;
        w3 = wi == 3 ? (w3 & m) | (b << sh) : w3;
        ++col;
        ++q;
    }
    u32x4 r;
    r.x = w0; r.y = w1; r.z = w2; r.w = w3;
    return r;
}

// v's bytes moved up by o (0..15): result byte j = v[j - o], zero below o.
__device__ __forceinline__ u32x4 place_at(u32x4 v, uint32_t o) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    return o == 0 ? v : funnel32(z, v, 16u - o);
}

__device__ __forceinline__ uint32_t pick_bytes(uint32_t a, uint32_t b, int32_t k) {
    // bytes below k from a, from k on from b (k in 0..4)
    if (k <= 0) return b;
    if (k >= 4) return a;
    const uint32_t m = (1u << (8 * k)) - 1u;
    return (a & m) | (b & ~m);
}

__device__ __forceinline__ u32x4 uslot_compose(const USlot &s, uint32_t c0) {
    u32x4 out = place_at(funnel32(s.a0, s.a1, s.sha), s.lo - c0);
    if (s.e1 < s.hi) {
        const u32x4 w = place_at(funnel32(s.b0, s.b1, s.shb), s.e1 - c0);
        const int32_t o = int32_t(s.e1 - c0);
        out.x = pick_bytes(out.x, w.x, o);
        out.y = pick_bytes(out.y, w.y, o - 4);
        out.z = pick_bytes(out.z, w.z, o - 8);
        out.w = pick_bytes(out.w, w.w, o - 12);
    }
    return out;
}

__device__ __forceinline__ void uslot_store(RS_GLOBAL unsigned char *slot, u32x4 v, const USlot &s, uint32_t c0) {
    if (s.lo == c0 && s.hi == c0 + 16u)
        store_vec((RS_GLOBAL u32x4 *)slot, v);
    else if (s.lo < s.hi)
        store_partial(slot, v, s.lo - c0, s.hi - c0);
}

// RF > 0: compile-time receiver count (vector-major stores up to 4
// receivers, as the aligned gather); RF == 0: runtime count.  SHORT: the
// group has segments shorter than 16 bytes.
template <int L, int RF, bool SHORT, int NPTR>
__device__ __forceinline__ void run_gather_u(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    const uint64_t *sp = reinterpret_cast<const uint64_t *>(rs_lds);
    const uint32_t *sst = reinterpret_cast<const uint32_t *>(rs_lds + 8u * kMaxSegs);
    const uint32_t *scol = reinterpret_cast<const uint32_t *>(rs_lds + 20u * kMaxSegs);
    const RS_CONST int32_t *fan = (const RS_CONST int32_t *)(a->fan + d.fan_off);
    const uint32_t nthr = blockDim.x, n = d.v1;
    const uint32_t nr = RF > 0 ? uint32_t(RF) : d.nfan;
    for (uint32_t ls = threadIdx.x; ls < n; ls += 2u * nthr) {
        const uint32_t c0 = 16u * ls, c1 = c0 + 16u * nthr;
        const bool has1 = ls + nthr < n;
        USlot s0, s1;
        uslot_load<L, SHORT>(d, sp, sst, scol, c0, s0);
        if (has1) uslot_load<L, SHORT>(d, sp, sst, scol, c1, s1);
        u32x4 o0 = uslot_compose(s0, c0);
        u32x4 o1 = has1 ? uslot_compose(s1, c1) : o0;
        if (SHORT) {
            if (s0.e2 < s0.hi) o0 = uslot_rest<L>(d, sp, sst, scol, s0, c0, o0);
            if (has1 && s1.e2 < s1.hi) o1 = uslot_rest<L>(d, sp, sst, scol, s1, c1, o1);
        }
        if constexpr (RF >= 1 && RF <= 4) {
#pragma unroll
            for (uint32_t r = 0; r < nr; ++r)
                uslot_store((RS_GLOBAL unsigned char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base + c0, o0, s0, c0);
            if (has1) {
#pragma unroll
                for (uint32_t r = 0; r < nr; ++r)
                    uslot_store((RS_GLOBAL unsigned char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base + c1, o1, s1,
                                c1);
            }
        } else if constexpr (RF > 4) {
#pragma unroll
            for (uint32_t r = 0; r < nr; ++r) {
                RS_GLOBAL unsigned char *dst =
                    (RS_GLOBAL unsigned char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base;
                uslot_store(dst + c0, o0, s0, c0);
                if (has1) uslot_store(dst + c1, o1, s1, c1);
            }
        } else {  // runtime receiver count
            for (uint32_t r = 0; r < nr; ++r) {
                RS_GLOBAL unsigned char *dst =
                    (RS_GLOBAL unsigned char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base;
                uslot_store(dst + c0, o0, s0, c0);
                if (has1) uslot_store(dst + c1, o1, s1, c1);
            }
        }
    }
}

typedef u32x4 u32x4_u __attribute__((aligned(1)));  // a 16-byte value at any byte address

// Unit gather (see desc.h): per lane, 16-byte units of the segments' rows,
// each one unaligned load and one unaligned store per receiver.  U units per
// lane per pass, loads first.  w: the unit's segment width (a segment under
// 16 bytes is one unit of w bytes).
template <int L, int U>
__device__ __forceinline__ void unit_addr(const Desc &d, const uint64_t *sp, const uint32_t *sst,
                                          const uint32_t *scol, const uint32_t *sunit, uint32_t v,
                                          const RS_GLOBAL unsigned char *&src, uint32_t &doff, uint32_t &w) {
    const uint32_t upr = d.vpr, ns = d.pad[1], rb = d.run;
    const uint32_t r = fastdiv(v, d.mul_vpr, d.sh_vpr);
    const uint32_t j = v - r * upr;
    uint32_t g = fastdiv(j, d.batch, d.pad[2]);
    if (g >= ns) g = ns - 1;
    while (g > 0 && j < sunit[g]) --g;
    while (g + 1 < ns && j >= sunit[g + 1]) ++g;
    w = (g + 1 < ns ? scol[g + 1] : rb) - scol[g];
    const uint32_t k16 = 16u * (j - sunit[g]);
    const uint32_t o = w < 16u ? 0u : k16 < w - 16u ? k16 : w - 16u;
    uint32_t i1, i2, i3;
    row_indices<L>(d, d.ss[0] + r, i1, i2, i3);
    src = (const RS_GLOBAL unsigned char *)(sp[g] + (i1 * sst[3 * g] + i2 * sst[3 * g + 1] + i3 * sst[3 * g + 2] + o));
    doff = (r - d.ss[1]) * rb + scol[g] + o;
}

#ifndef RS_UNIT_U
#define RS_UNIT_U 2
#endif

// The n (< 16) bytes at q as the low bytes of a 16-byte value: the one or
// two aligned words that hold them, funnel-shifted (an aligned word holding
// one byte of a buffer lies inside the buffer's allocation).
__device__ __forceinline__ u32x4 load_short(const RS_GLOBAL unsigned char *q, uint32_t n) {
    const uint64_t a = uint64_t(q);
    const uint32_t sh = uint32_t(a) & 15u;
    const RS_GLOBAL u32x4 *w = (const RS_GLOBAL u32x4 *)(a & ~uint64_t(15));
    const u32x4 z = {0u, 0u, 0u, 0u};
    const u32x4 w0 = w[0];
    const u32x4 w1 = sh + n > 16u ? w[1] : z;
    return funnel32(w0, w1, sh);
}

// The low n (< 16) bytes of v to q, one byte store each.
__device__ __forceinline__ void store_short(RS_GLOBAL unsigned char *q, u32x4 v, uint32_t n) {
    const uint32_t x[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (uint32_t i = 0; i < 15u; ++i)
        if (i < n) q[i] = (unsigned char)(x[i >> 2] >> (8u * (i & 3u)));
}

// SHORT: the group has segments shorter than 16 bytes.  Each is one unit,
// skipped by the main loop and moved afterwards in one pass over the
// chunk's short units (load_short / store_short), so the waves of the main
// loop never branch to the byte path.
template <int L, bool SHORT, int NPTR>
__device__ __forceinline__ void run_gather_unit(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    constexpr int U = RS_UNIT_U;  // units per lane per pass, loads first
    const uint64_t *sp = reinterpret_cast<const uint64_t *>(rs_lds);
    const uint32_t *sst = reinterpret_cast<const uint32_t *>(rs_lds + 8u * kMaxSegs);
    const uint32_t *scol = reinterpret_cast<const uint32_t *>(rs_lds + 20u * kMaxSegs);
    const uint32_t *sunit = reinterpret_cast<const uint32_t *>(rs_lds + 24u * kMaxSegs);
    const RS_CONST int32_t *fan = (const RS_CONST int32_t *)(a->fan + d.fan_off);
    const uint32_t nthr = blockDim.x;
    for (uint32_t v = d.v0 + threadIdx.x; v < d.v1; v += U * nthr) {
        u32x4 x[U];
        uint32_t doff[U], w[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t vu = v + uint32_t(u) * nthr;
            if (vu < d.v1) {
                const RS_GLOBAL unsigned char *src;
                unit_addr<L, U>(d, sp, sst, scol, sunit, vu, src, doff[u], w[u]);
                if (!SHORT || w[u] >= 16u) x[u] = *(const RS_GLOBAL u32x4_u *)src;
            }
        }
        for (uint32_t r = 0; r < d.nfan; ++r) {
            RS_GLOBAL unsigned char *dst = (RS_GLOBAL unsigned char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (v + uint32_t(u) * nthr >= d.v1 || (SHORT && w[u] < 16u)) continue;
                store_vec((RS_GLOBAL u32x4_u *)(dst + doff[u]), x[u]);
            }
        }
    }
    if constexpr (SHORT) {
        // the chunk's short units: (row, short segment) pairs of its rows
        const uint32_t *sshort = reinterpret_cast<const uint32_t *>(rs_lds + 28u * kMaxSegs);
        const uint32_t nsh = *reinterpret_cast<const uint32_t *>(rs_lds + 32u * kMaxSegs);
        const uint32_t ns = d.pad[1], rb = d.run;
        const uint32_t r0 = fastdiv(d.v0, d.mul_vpr, d.sh_vpr), r1 = fastdiv(d.v1 - 1u, d.mul_vpr, d.sh_vpr);
        const uint32_t total = (r1 - r0 + 1u) * nsh;
        for (uint32_t i = threadIdx.x; i < total; i += nthr) {
            const uint32_t rr = i / nsh, g = sshort[i - rr * nsh], r = r0 + rr;
            const uint32_t vu = r * d.vpr + sunit[g];
            if (vu < d.v0 || vu >= d.v1) continue;
            const uint32_t ws = (g + 1 < ns ? scol[g + 1] : rb) - scol[g];
            uint32_t i1, i2, i3;
            row_indices<L>(d, d.ss[0] + r, i1, i2, i3);
            const RS_GLOBAL unsigned char *q =
                (const RS_GLOBAL unsigned char *)(sp[g] + (i1 * sst[3 * g] + i2 * sst[3 * g + 1] + i3 * sst[3 * g + 2]));
            const u32x4 y = load_short(q, ws);
            const uint32_t off = (r - d.ss[1]) * rb + scol[g];
            for (uint32_t k = 0; k < d.nfan; ++k)
                store_short((RS_GLOBAL unsigned char *)a->ptr[a->nsrc + uint32_t(fan[k])] + d.dst_base + off, y, ws);
        }
    }
}


template <int L, int NPTR>
__device__ __forceinline__ void run_gather_u_fan(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    if (d.ds[0] & kUShortSegs) {
        // segments under 16 bytes: compile-time receiver counts up to 4
        // (measured at fan-out 4: 403 -> 389 us against one runtime-count form)
        switch (d.nfan) {
            case 1: run_gather_u<L, 1, true>(d, a); return;
            case 2: run_gather_u<L, 2, true>(d, a); return;
            case 3: run_gather_u<L, 3, true>(d, a); return;
            case 4: run_gather_u<L, 4, true>(d, a); return;
            default: run_gather_u<L, 0, true>(d, a); return;
        }
    }
    switch (d.nfan) {
        case 1: run_gather_u<L, 1, false>(d, a); break;
        case 2: run_gather_u<L, 2, false>(d, a); break;
        case 3: run_gather_u<L, 3, false>(d, a); break;
        case 4: run_gather_u<L, 4, false>(d, a); break;
        case 5: run_gather_u<L, 5, false>(d, a); break;
        case 6: run_gather_u<L, 6, false>(d, a); break;
        case 7: run_gather_u<L, 7, false>(d, a); break;
        case 8: run_gather_u<L, 8, false>(d, a); break;
        default: run_gather_u<L, 0, false>(d, a); break;
    }
}

template <int NPTR>
__global__ __launch_bounds__(256) void reshard_gather_u_kernel(KArgs<NPTR> args) {
    const RS_CONST KArgs<NPTR> *a = (const RS_CONST KArgs<NPTR> *)__builtin_amdgcn_kernarg_segment_ptr();
    const uint32_t b = blockIdx.x;
    const uint32_t idx = a->per_xcd ? (b & 7u) * a->per_xcd + (b >> 3) : grouped_chunk(b);
    if (idx >= a->ndesc) return;
    const Desc d = load_desc(a, idx);
    stage_segments_u(d, a);
    __syncthreads();
    switch (kind_levels(d.kind)) {
        case 1: run_gather_u_fan<1>(d, a); break;
        case 2: run_gather_u_fan<2>(d, a); break;
        default: run_gather_u_fan<3>(d, a); break;
    }
}

// Tile transpose (see desc.h): per tile, a load phase (rows of the tile,
// contiguous in the sender's buffer, into LDS: 16-byte vectors where the
// rows are aligned, else element by element) and a store phase (columns of
// the tile, contiguous in the receivers' buffers: each lane assembles one
// 16-byte vector from 16 / ES rows of one column and stores it to every
// receiver).  Lanes 8k .. 8k + 7 cover one row (one column) of 128 bytes,
// so a wave moves 8 whole cache lines per instruction on both sides.
template <int ES>
__device__ __forceinline__ void tile_put(unsigned char *lds, uint32_t off, u32x4 v) {
    *reinterpret_cast<u32x4 *>(lds + off) = v;
}

template <int ES>
__device__ __forceinline__ u32x4 tile_column(const unsigned char *lds, uint32_t b0, uint32_t a) {
    const uint32_t c = (a * ES) >> 4, o = (a * ES) & 15u;
    if constexpr (ES == 8) {
        u32x4 y;
        const u32x2 lo = *reinterpret_cast<const u32x2 *>(lds + tile_lds(b0, c, o, ES));
        const u32x2 hi = *reinterpret_cast<const u32x2 *>(lds + tile_lds(b0 + 1, c, o, ES));
        y.x = lo.x; y.y = lo.y; y.z = hi.x; y.w = hi.y;
        return y;
    } else if constexpr (ES == 4) {
        u32x4 y;
        y.x = *reinterpret_cast<const uint32_t *>(lds + tile_lds(b0, c, o, ES));
        y.y = *reinterpret_cast<const uint32_t *>(lds + tile_lds(b0 + 1, c, o, ES));
        y.z = *reinterpret_cast<const uint32_t *>(lds + tile_lds(b0 + 2, c, o, ES));
        y.w = *reinterpret_cast<const uint32_t *>(lds + tile_lds(b0 + 3, c, o, ES));
        return y;
    } else {
        uint32_t w[4];
#pragma unroll
        for (uint32_t q = 0; q < 4; ++q) {
            uint32_t acc = 0;
#pragma unroll
            for (uint32_t e = 0; e < 4 / ES; ++e) {
                const uint32_t r = b0 + q * (4 / ES) + e;
                uint32_t x;
                if constexpr (ES == 2) x = *reinterpret_cast<const uint16_t *>(lds + tile_lds(r, c, o, ES));
                else x = lds[tile_lds(r, c, o, ES)];
                acc |= x << (8u * ES * e);
            }
            w[q] = acc;
        }
        u32x4 y;
        y.x = w[0]; y.y = w[1]; y.z = w[2]; y.w = w[3];
        return y;
    }
}

template <int ES> struct Elem;
template <> struct Elem<1> { typedef unsigned char T; };
template <> struct Elem<2> { typedef unsigned short T; };
template <> struct Elem<4> { typedef unsigned int T; };
template <> struct Elem<8> { typedef unsigned long long T; };

// The first n (< 16 / ES) elements at q, one load each, packed into a
// 16-byte value (the rest zero).  Unrolled with constant indices, so the
// value stays in registers.
template <int ES>
__device__ __forceinline__ u32x4 load_elems(const RS_GLOBAL unsigned char *q, uint32_t n) {
    typedef typename Elem<ES>::T E;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (uint32_t e = 0; e < 16u / ES; ++e) {
        if (e < n) {
            const E v = ((const RS_GLOBAL E *)q)[e];
            if constexpr (ES == 8) {
                w[2 * e] = uint32_t(v);
                w[2 * e + 1] = uint32_t(uint64_t(v) >> 32);
            } else {
                w[(e * ES) / 4] |= uint32_t(v) << (8u * ((e * ES) % 4));
            }
        }
    }
    u32x4 x;
    x.x = w[0]; x.y = w[1]; x.z = w[2]; x.w = w[3];
    return x;
}

// Store the first n (< 16 / ES) elements of y at q, one store each.
template <int ES>
__device__ __forceinline__ void store_elems(RS_GLOBAL unsigned char *q, u32x4 y, uint32_t n) {
    typedef typename Elem<ES>::T E;
    const uint32_t w[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
    for (uint32_t e = 0; e < 16u / ES; ++e) {
        if (e < n) {
            E v;
            if constexpr (ES == 8) v = E(w[2 * e]) | (E(w[2 * e + 1]) << 32);
            else v = E(w[(e * ES) / 4] >> (8u * ((e * ES) % 4)));
            ((RS_GLOBAL E *)q)[e] = v;
        }
    }
}

// G: tile-row vectors per lane loaded before any is written to LDS.
// Measured on an fp16 [8,2048,12288] transpose: 4 is 4 % faster than 1 at
// fan-out 1, where reads are half of a tile's traffic; at fan-out 4 it
// measured from 2 % slower to equal, so only one receiver uses it.
template <int ES, uint32_t G, int NPTR>
__device__ __forceinline__ void run_transpose(const Desc &d, const RS_CONST KArgs<NPTR> *a) {
    constexpr uint32_t T = kTileBytes / ES, V = 16u / ES;
    const uint32_t TR = tile_rows(ES, d.kind), SL = TR * ES / 16u;  // tile rows; 16-byte slots per column
    unsigned char *lds = rs_lds;
    const RS_GLOBAL unsigned char *src = (const RS_GLOBAL unsigned char *)a->ptr[d.src_buf] + d.src_base;
    const RS_CONST int32_t *fan = (const RS_CONST int32_t *)(a->fan + d.fan_off);
    const bool ald = (d.kind & kTAlignLoad) != 0, ast = (d.kind & kTAlignStore) != 0;
    const uint32_t nthr = blockDim.x, tid = threadIdx.x;
    const uint32_t wl2 = tile_wide_log2(d.kind);
    for (uint32_t t = d.v0; t < d.v1; ++t) {
        const TileAt at = tile_offsets(d, t, ES);
        const uint32_t na = d.run - at.ta * T < T ? d.run - at.ta * T : T;
        const uint32_t nb = d.batch - at.tb * TR < TR ? d.batch - at.tb * TR : TR;
        for (uint32_t i0 = tid; i0 < TR * 8u; i0 += G * nthr) {
            u32x4 x[G];
#pragma unroll
            for (uint32_t k = 0; k < G; ++k) {
                const uint32_t i = i0 + k * nthr, r = i >> 3, c = i & 7u;
                if (i >= TR * 8u || r >= nb) continue;
                const uint32_t a0 = c * V;
                const uint32_t nv = a0 < na ? (na - a0 < V ? na - a0 : V) : 0u;
                const RS_GLOBAL unsigned char *q = src + (at.src + r * d.ss[0] + c * 16u);
                if (nv == V && ald) x[k] = load_vec((const RS_GLOBAL u32x4 *)q);
                else x[k] = load_elems<ES>(q, nv);
            }
#pragma unroll
            for (uint32_t k = 0; k < G; ++k) {
                const uint32_t i = i0 + k * nthr, r = i >> 3, c = i & 7u;
                if (i < TR * 8u && r < nb) tile_put<ES>(lds, tile_lds(r, c, 0, ES), x[k]);
            }
        }
        __syncthreads();
        for (uint32_t i = tid; i < T * SL; i += nthr) {
            const uint32_t aa = i >> (3u + wl2), j = i & (SL - 1u);
            if (aa >= na) continue;
            const uint32_t b0 = j * V;
            const uint32_t nv = b0 < nb ? (nb - b0 < V ? nb - b0 : V) : 0u;
            if (nv == 0) continue;
            const u32x4 y = tile_column<ES>(lds, b0, aa);
            const uint32_t off = at.dst + aa * d.ds[0] + j * 16u;
            if (nv == V && ast) {
                for (uint32_t r = 0; r < d.nfan; ++r) {
                    RS_GLOBAL char *dst = (RS_GLOBAL char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base;
                    store_vec((RS_GLOBAL u32x4 *)(dst + off), y);
                }
            } else {
                for (uint32_t r = 0; r < d.nfan; ++r)
                    store_elems<ES>((RS_GLOBAL unsigned char *)a->ptr[a->nsrc + uint32_t(fan[r])] + d.dst_base + off,
                                    y, nv);
            }
        }
        __syncthreads();
    }
}

template <int NPTR>
__global__ __launch_bounds__(256) void reshard_transpose_kernel(KArgs<NPTR> args) {
    const RS_CONST KArgs<NPTR> *a = (const RS_CONST KArgs<NPTR> *)__builtin_amdgcn_kernarg_segment_ptr();
    const uint32_t b = blockIdx.x;
    const uint32_t idx = a->per_xcd ? (b & 7u) * a->per_xcd + (b >> 3) : b;
    if (idx >= a->ndesc) return;
    const Desc d = load_desc(a, idx);
    if (d.nfan == 1) {
        switch (d.kind & 0xFu) {
            case 0: run_transpose<1, 4>(d, a); break;
            case 1: run_transpose<2, 4>(d, a); break;
            case 2: run_transpose<4, 4>(d, a); break;
            default: run_transpose<8, 4>(d, a); break;
        }
    } else {
        switch (d.kind & 0xFu) {
            case 0: run_transpose<1, 1>(d, a); break;
            case 1: run_transpose<2, 1>(d, a); break;
            case 2: run_transpose<4, 1>(d, a); break;
            default: run_transpose<8, 1>(d, a); break;
        }
    }
}

// Unit-gather chunks in their own kernel, so the slot kernel keeps its
// registers (measured: sharing one kernel slowed the slot path 12-27 %).
template <int NPTR>
__global__ __launch_bounds__(256) void reshard_gather_unit_kernel(KArgs<NPTR> args) {
    const RS_CONST KArgs<NPTR> *a = (const RS_CONST KArgs<NPTR> *)__builtin_amdgcn_kernarg_segment_ptr();
    const uint32_t b = blockIdx.x;
    const uint32_t idx = a->per_xcd ? (b & 7u) * a->per_xcd + (b >> 3) : grouped_chunk(b);
    if (idx >= a->ndesc) return;
    const Desc d = load_desc(a, idx);
    if (d.ds[0] & kUShortSegs) {  // uniform: clear the short-segment count first
        if (threadIdx.x == 0) *reinterpret_cast<uint32_t *>(rs_lds + 32u * kMaxSegs) = 0u;
        __syncthreads();
    }
    stage_segments_u<NPTR, true>(d, a);
    __syncthreads();
    if (d.ds[0] & kUShortSegs) {
        switch (kind_levels(d.kind)) {
            case 1: run_gather_unit<1, true>(d, a); break;
            case 2: run_gather_unit<2, true>(d, a); break;
            default: run_gather_unit<3, true>(d, a); break;
        }
        return;
    }
    switch (kind_levels(d.kind)) {
        case 1: run_gather_unit<1, false>(d, a); break;
        case 2: run_gather_unit<2, false>(d, a); break;
        default: run_gather_unit<3, false>(d, a); break;
    }
}

// Realignment chunks run in their own kernel so their register use does not
// bound the direct kernel's occupancy.  STAGE: through LDS, else shifted loads.
template <int NPTR, bool STAGE>
__global__ __launch_bounds__(256) void reshard_realign_kernel(KArgs<NPTR> args) {
    const RS_CONST KArgs<NPTR> *a = (const RS_CONST KArgs<NPTR> *)__builtin_amdgcn_kernarg_segment_ptr();
    const uint32_t b = blockIdx.x;
    const uint32_t idx = a->per_xcd ? (b & 7u) * a->per_xcd + (b >> 3) : b;
    if (idx >= a->ndesc) return;
    const Desc d = load_desc(a, idx);
    if (STAGE) {
        switch (kind_levels(d.kind)) {
            case 1: run_realign<1>(d, a); break;
            case 2: run_realign<2>(d, a); break;
            default: run_realign<3>(d, a); break;
        }
    } else {
        switch (kind_levels(d.kind)) {
            case 1: run_shift<1>(d, a); break;
            case 2: run_shift<2>(d, a); break;
            default: run_shift<3>(d, a); break;
        }
    }
}

// ------------------------------------------------------------------ host

namespace {

reshard_status_t hip_fail(const char *what, hipError_t e) {
    return fail(RESHARD_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Upload [descs | fan] to the current device once; returns the device pointer.
reshard_status_t device_table(const Plan &p, int dev, const Desc **descs, const int32_t **fan, const Seg **segs) {
    if (dev < 0 || dev >= Plan::kMaxHipDevices)
        return fail(RESHARD_EUNSUPPORTED, "HIP device ordinal " + std::to_string(dev) + " above the plan's limit");
    std::lock_guard<std::mutex> lock(p.mu);
    const size_t dbytes = p.descs.size() * sizeof(Desc);
    const size_t fbytes = p.fan.size() * sizeof(int32_t);
    const size_t soff = (dbytes + fbytes + 15) & ~size_t(15);
    const size_t sbytes = p.segs.size() * sizeof(Seg);
    if (!p.d_table[dev]) {
        void *mem = nullptr;
        hipError_t e = hipMalloc(&mem, soff + sbytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(RESHARD_ENOMEM, std::string("hipMalloc of the descriptor table: ") + hipGetErrorString(e));
        }
        e = hipMemcpy(mem, p.descs.data(), dbytes, hipMemcpyHostToDevice);
        if (e == hipSuccess && fbytes)
            e = hipMemcpy(static_cast<char *>(mem) + dbytes, p.fan.data(), fbytes, hipMemcpyHostToDevice);
        if (e == hipSuccess && sbytes)
            e = hipMemcpy(static_cast<char *>(mem) + soff, p.segs.data(), sbytes, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            (void)hipFree(mem);
            return hip_fail("upload of the descriptor table", e);
        }
        p.d_table[dev] = mem;
    }
    *descs = static_cast<const Desc *>(p.d_table[dev]);
    *fan = reinterpret_cast<const int32_t *>(static_cast<const char *>(p.d_table[dev]) + dbytes);
    *segs = reinterpret_cast<const Seg *>(static_cast<const char *>(p.d_table[dev]) + soff);
    return RESHARD_OK;
}

template <typename K, typename A>
reshard_status_t launch_one(K kernel, A a, uint32_t ndesc, bool remap, uint32_t block, uint32_t lds,
                            hipStream_t stream, uint32_t grid_multiple = 1) {
    a.ndesc = ndesc;
    uint32_t grid = (ndesc + grid_multiple - 1u) / grid_multiple * grid_multiple;  // ndesc < 2^24
    a.per_xcd = 0;
    if (remap) {
        a.per_xcd = (ndesc + 7u) / 8u;
        grid = a.per_xcd * 8u;
    }
    if (lds > 64u * 1024u) {
        // above the default dynamic-LDS limit; raising it is idempotent
        const hipError_t ea = hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                                                  hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
        if (ea != hipSuccess) return hip_fail("raising the kernel's LDS limit", ea);
    }
    hipLaunchKernelGGL(kernel, dim3(grid), dim3(block), lds, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail("kernel launch", e);
    return RESHARD_OK;
}

// LDS reservation (unused by the direct kernel; the gather kernels' segment
// tables fit inside it) that caps resident workgroups per CU.  The CU's
// 160 KiB of LDS is handed out as two 80 KiB halves and a workgroup's
// reservation must fit in one half (measured occupancy: reservations for 3
// or 5 workgroups per CU leave 2 or 4 resident), so the cap is an even
// number of workgroups: n per half.
uint32_t lds_for_per_half(uint32_t n) {
    if (n < 1u) n = 1u;
    return n >= 16u ? 0u : (80u * 1024u / n) & ~1023u;
}

// ... for at most `waves` waves per CU, never below 2 workgroups.
uint32_t residency_lds(uint32_t waves, uint32_t block) {
    return lds_for_per_half(waves / (2u * (block / 64u ? block / 64u : 1u)));
}

template <int NPTR>
reshard_status_t launch(const Plan &p, const Desc *descs, const int32_t *fan, const Seg *segs,
                        void *const *src_ptrs, void *const *dst_ptrs, hipStream_t stream) {
    KArgs<NPTR> a;
    a.descs = descs;
    a.fan = fan;
    a.segs = segs;
    a.ndesc = 0;
    a.nsrc = uint32_t(p.src.ndev);
    a.per_xcd = 0;
    a.pad = 0;
    for (int64_t k = 0; k < p.src.ndev; ++k) a.ptr[k] = src_ptrs[k];
    for (int64_t k = 0; k < p.dst.ndev; ++k) a.ptr[p.src.ndev + k] = dst_ptrs[k];
    const bool remap = (p.flags & RESHARD_XCD_REMAP) != 0;
    const uint32_t block = uint32_t(p.tuning.block_threads);
    // Direct chunks at fan-out 2 run 512-thread workgroups unless the caller
    // chose a block size: a 16 KiB chunk is then one batch of loads before
    // its stores, on half as many resident chunks (measured 1.5-4 % faster
    // on four fan-out-2 tensors, slower at fan-out 1, 4 and 8).
    const uint32_t dblock = p.tuning.block_is_default && p.direct_fanout == 2 ? 512u : block;
    // Residency cap of the direct and gather kernels: the caller's (rounded
    // down to an even number of workgroups), else chosen from the kernel's
    // fan-out (measured with buffers that are not cache-resident): direct
    // chunks 16 waves per CU at fan-out <= 2, 8 above; gather chunks about
    // 64 receiver write streams per CU (64 / fan-out waves, at least 8).
    const uint32_t user_lds =
        p.tuning.max_wgs_per_cu ? lds_for_per_half(uint32_t(p.tuning.max_wgs_per_cu) / 2u) : 0u;
    const uint32_t cap_lds =
        p.tuning.cap_is_default ? residency_lds(p.direct_fanout <= 2 ? 16u : 8u, dblock) : user_lds;
    const uint32_t n_direct = uint32_t(p.n_direct), n_gather = uint32_t(p.n_gather);
    const uint32_t n_gather_u = uint32_t(p.n_gather_u);
    const uint32_t n_transpose = uint32_t(p.n_transpose);
    const uint32_t n_realign = uint32_t(p.descs.size() - p.n_direct - p.n_gather - p.n_gather_u - p.n_transpose);
    const uint32_t n_phase1 = uint32_t(p.n_phase1);
    if (n_phase1) {
        const reshard_status_t st = launch_one(reshard_kernel<NPTR>, a, n_phase1, remap, dblock, cap_lds, stream);
        if (st != RESHARD_OK) return st;
    }
    if (n_direct > n_phase1) {  // second phase, stream-ordered after the first
        a.descs = descs + n_phase1;
        const reshard_status_t st =
            launch_one(reshard_kernel<NPTR>, a, n_direct - n_phase1, remap, dblock, cap_lds, stream);
        if (st != RESHARD_OK) return st;
    }
    if (n_gather) {
        uint32_t gcap_lds = user_lds;
        if (p.tuning.cap_is_default) {
            const uint32_t fan = uint32_t(p.gather_fanout > 0 ? p.gather_fanout : 1);
            gcap_lds = residency_lds(64u / fan > 8u ? 64u / fan : 8u, block);
        }
        const uint32_t need = (12u + 8u) * kMaxSegs;
        const uint32_t glds = gcap_lds > need ? gcap_lds : need;
        a.descs = descs + n_direct;
        const reshard_status_t st = launch_one(reshard_gather_kernel<NPTR>, a, n_gather, remap, block, glds, stream);
        if (st != RESHARD_OK) return st;
    }
    // the unaligned row-gather section: slot chunks, then unit chunks
    const uint32_t n_unit = uint32_t(p.n_unit), n_slot = n_gather_u - n_unit;
    // Rows gathered from several senders: about 64 receiver write streams
    // per CU, as the aligned gather.  One sender per row (rows in runs, or
    // whole rows in another phase) reads like the direct kernel and wants
    // its caps: measured uncapped best at fan-out 1, 16 waves at 2 (10 %
    // faster than uncapped), 8 at 4 (12 % faster than 16) -- unless most
    // chunks are cut short by their runs: each then makes one short pass,
    // its latency is not hidden, and 32 waves are best (8 KiB runs at
    // fan-out 4: 141 against 197 us).  Segments under 16 bytes (the slow
    // slot path) want 32 waves too (fan-out 4: 382 against 390 us).
    auto gather_u_lds = [&](int64_t fanout, int64_t segs, bool more_waves) {
        if (!p.tuning.cap_is_default) return user_lds;
        const uint32_t fan = uint32_t(fanout > 0 ? fanout : 1);
        uint32_t waves = 64u / fan > 8u ? 64u / fan : 8u;
        if (segs == 1) waves = fan <= 1 ? 32u : fan == 2 ? 16u : 8u;
        if (more_waves && waves < 32u) waves = 32u;
        return residency_lds(waves, block < 256u ? block : 256u);
    };
    if (n_slot) {
        const bool short_chunks = p.gather_u_segs == 1 && 4 * p.gather_u_bytes < 3 * p.gather_u_room;
        const bool short_segs = p.gather_u_short && p.gather_u_fanout <= 4;  // measured up to fan-out 4
        const uint32_t ulds = gather_u_lds(p.gather_u_fanout, p.gather_u_segs, short_chunks || short_segs);
        a.descs = descs + n_direct + n_gather;
        const reshard_status_t st = launch_one(reshard_gather_u_kernel<NPTR>, a, n_slot, remap,
                                               block < 256u ? block : 256u,
                                               ulds > kGatherULds ? ulds : kGatherULds, stream, 8u * kUGroup);
        if (st != RESHARD_OK) return st;
    }
    if (n_unit) {
        const uint32_t ulds = gather_u_lds(p.unit_fanout, p.unit_segs, false);
        a.descs = descs + n_direct + n_gather + n_slot;
        const reshard_status_t st = launch_one(reshard_gather_unit_kernel<NPTR>, a, n_unit, remap,
                                               block < 256u ? block : 256u, ulds > kUnitLds ? ulds : kUnitLds,
                                               stream, 8u * kUGroup);
        if (st != RESHARD_OK) return st;
    }
    if (n_transpose) {
        // the widest tile of the plan (rows of kTileBytes) in LDS;
        // no residency cap
        a.descs = descs + n_direct + n_gather + n_gather_u;
        const uint32_t tblock = block < 256u ? block : 256u;
        const uint32_t lds = p.transpose_rows * kTileBytes;
        const reshard_status_t st =
            launch_one(reshard_transpose_kernel<NPTR>, a, n_transpose, remap, tblock, lds, stream);
        if (st != RESHARD_OK) return st;
    }
    if (n_realign) {
        a.descs = descs + n_direct + n_gather + n_gather_u + n_transpose;
        // Realignment kernels hide their load -> shift -> store latency with
        // resident workgroups: no residency cap (measured: capping at 12
        // waves per CU halves their throughput).  Staging takes its LDS.
        const uint32_t need = (p.lds_bytes + 1023u) & ~1023u;
        const uint32_t rblock = block < 256u ? block : 256u;  // the realignment kernel's bound
        const reshard_status_t st =
            (p.flags & RESHARD_LDS_STAGING)
                ? launch_one(reshard_realign_kernel<NPTR, true>, a, n_realign, remap, rblock, need, stream)
                : launch_one(reshard_realign_kernel<NPTR, false>, a, n_realign, remap, rblock, 0u, stream);
        if (st != RESHARD_OK) return st;
    }
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

extern "C" reshard_status_t reshard_plan_upload(const reshard_plan_t *plan) {
    return rs::guarded([&]() -> reshard_status_t {
        using namespace rs;
        const Plan *p = reinterpret_cast<const Plan *>(plan);
        if (!p) return fail(RESHARD_EINVAL, "NULL plan");
        if (p->descs.empty()) return RESHARD_OK;
        int dev = -1;
        const hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return fail(RESHARD_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
        const Desc *descs = nullptr;
        const int32_t *fan = nullptr;
        const Seg *segs = nullptr;
        return device_table(*p, dev, &descs, &fan, &segs);
    });
}

namespace rs {
namespace {

// The caller's buffers: every non-empty shard has a pointer, aligned as the
// plan's vectors need.
reshard_status_t check_buffers(const Plan *p, void *const *src_ptrs, void *const *dst_ptrs) {
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
    return RESHARD_OK;
}

reshard_status_t launch_any(const Plan &p, const Desc *descs, const int32_t *fan, const Seg *segs,
                            void *const *src_ptrs, void *const *dst_ptrs, hipStream_t s) {
    if (p.src.ndev + p.dst.ndev <= 64) return launch<64>(p, descs, fan, segs, src_ptrs, dst_ptrs, s);
    return launch<RESHARD_MAX_BUFFERS>(p, descs, fan, segs, src_ptrs, dst_ptrs, s);
}

}  // namespace

// Scratch of reshard_execute_noalloc: the plan's descriptor, receiver and
// segment tables are copied here (same layout as the plan's own device
// table) instead of into memory the library allocates.  Each device holds
// one copy for the life of the process.  Host code never passes the array's
// name to a kernel or a copy: it passes the device address that
// hipGetSymbolAddress returned on that device.
static __device__ __align__(256) unsigned char scratch[RESHARD_NOALLOC_MAX_TABLE_BYTES];

namespace {

struct ScratchState {
    std::mutex mu;
    void *addr[Plan::kMaxHipDevices] = {};           // device address of `scratch`, per device
    uint64_t plan[Plan::kMaxHipDevices] = {};        // serial of the plan whose tables it holds
    void *stream[Plan::kMaxHipDevices] = {};         // the stream that copy was ordered on
};

ScratchState &scratch_state() {
    static ScratchState st;
    return st;
}

}  // namespace
}  // namespace rs

extern "C" reshard_status_t reshard_execute(const reshard_plan_t *plan, void *const *src_ptrs,
                                            void *const *dst_ptrs, void *stream) {
    return rs::guarded([&]() -> reshard_status_t {
        using namespace rs;
        const Plan *p = reinterpret_cast<const Plan *>(plan);
        reshard_status_t st = check_buffers(p, src_ptrs, dst_ptrs);
        if (st != RESHARD_OK) return st;
        if (p->descs.empty()) return RESHARD_OK;
        int dev = -1;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return fail(RESHARD_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
        const Desc *descs = nullptr;
        const int32_t *fan = nullptr;
        const Seg *segs = nullptr;
        st = device_table(*p, dev, &descs, &fan, &segs);
        if (st != RESHARD_OK) return st;
        return launch_any(*p, descs, fan, segs, src_ptrs, dst_ptrs, static_cast<hipStream_t>(stream));
    });
}

extern "C" reshard_status_t reshard_execute_noalloc(const reshard_plan_t *plan, void *const *src_ptrs,
                                                    void *const *dst_ptrs, void *stream) {
    return rs::guarded([&]() -> reshard_status_t {
        using namespace rs;
        const Plan *p = reinterpret_cast<const Plan *>(plan);
        reshard_status_t st = check_buffers(p, src_ptrs, dst_ptrs);
        if (st != RESHARD_OK) return st;
        if (p->descs.empty()) return RESHARD_OK;
        const size_t dbytes = p->descs.size() * sizeof(Desc);
        const size_t fbytes = p->fan.size() * sizeof(int32_t);
        const size_t soff = (dbytes + fbytes + 15) & ~size_t(15);
        const size_t total = soff + p->segs.size() * sizeof(Seg);
        if (total > size_t(RESHARD_NOALLOC_MAX_TABLE_BYTES))
            return fail(RESHARD_EUNSUPPORTED, "the plan's tables take " + std::to_string(total) +
                                                  " bytes; reshard_execute_noalloc holds at most " +
                                                  std::to_string(RESHARD_NOALLOC_MAX_TABLE_BYTES) +
                                                  " (use reshard_execute, or larger chunks)");
        int dev = -1;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return fail(RESHARD_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
        if (dev < 0 || dev >= Plan::kMaxHipDevices)
            return fail(RESHARD_EUNSUPPORTED, "HIP device ordinal " + std::to_string(dev) + " above the limit");
        hipStream_t s = static_cast<hipStream_t>(stream);
        char *base = nullptr;
        {
            ScratchState &ss = scratch_state();
            std::lock_guard<std::mutex> lock(ss.mu);
            if (!ss.addr[dev]) {
                void *addr = nullptr;
                e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
                if (e != hipSuccess || !addr) {
                    (void)hipGetLastError();
                    return fail(RESHARD_EHIP, std::string("hipGetSymbolAddress of the scratch table: ") +
                                                  hipGetErrorString(e));
                }
                ss.addr[dev] = addr;
            }
            base = static_cast<char *>(ss.addr[dev]);
            // The tables are copied on the call's stream, so its kernels see
            // them; the same plan executed again on the same stream finds
            // them in place.  Nothing in the scratch must start at zero: the
            // kernels only read what the copy wrote.
            if (ss.plan[dev] != p->serial || ss.stream[dev] != stream) {
                ss.plan[dev] = 0;
                e = hipMemcpyAsync(base, p->descs.data(), dbytes, hipMemcpyHostToDevice, s);
                if (e == hipSuccess && fbytes)
                    e = hipMemcpyAsync(base + dbytes, p->fan.data(), fbytes, hipMemcpyHostToDevice, s);
                if (e == hipSuccess && !p->segs.empty())
                    e = hipMemcpyAsync(base + soff, p->segs.data(), total - soff, hipMemcpyHostToDevice, s);
                if (e != hipSuccess) {
                    (void)hipGetLastError();
                    return fail(RESHARD_EHIP, std::string("copy of the plan's tables into the scratch: ") +
                                                  hipGetErrorString(e));
                }
                ss.plan[dev] = p->serial;
                ss.stream[dev] = stream;
            }
        }
        return launch_any(*p, reinterpret_cast<const Desc *>(base), reinterpret_cast<const int32_t *>(base + dbytes),
                          reinterpret_cast<const Seg *>(base + soff), src_ptrs, dst_ptrs, s);
    });
}
