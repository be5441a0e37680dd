// Host-side fuzz driver for the planner, the host interpreter, the
// scheduler and the pipeline model, built with AddressSanitizer and
// UndefinedBehaviorSanitizer (no GPU code).  Random tensors (rank 1..4,
// extents 0..40, element sizes 1/2/4/8), meshes (1..3 axes of 1..4 devices)
// and specs, under every lowering flag and several tunings; each plan runs
// through the host interpreter on buffers of exactly the shard sizes, so any
// access outside them is reported.  Then plans only, at sizes far beyond
// this host's memory.  Prints "ok <plans>" on success.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <utility>
#include <vector>

#include "reshard.h"

namespace rs {
struct Plan;
// the device-table release lives with the kernels; host-only builds have none
void release_device_table(const Plan &) {}
}  // namespace rs

static uint64_t rng_state = 0x243F6A8885A308D3ull;
static uint32_t rnd(uint32_t n) {  // xorshift64*, n > 0
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return uint32_t((rng_state * 0x2545F4914F6CDD1Dull) >> 32) % n;
}

static std::string random_spec(int ndim, int mesh_ndim) {
    std::vector<std::vector<int>> axes(ndim);
    for (int a = 0; a < mesh_ndim; ++a)
        if (rnd(3)) axes[rnd(ndim)].push_back(a);  // each mesh axis on at most one dim, or replicated
    std::string s;
    for (int d = 0; d < ndim; ++d) {
        if (axes[d].empty()) {
            s += "R";
        } else {
            s += "S^{";
            for (int a : axes[d]) s += char('0' + a);
            s += "}";
        }
    }
    return s;
}

int main(int argc, char **argv) {
    const int iters = argc > 1 ? atoi(argv[1]) : 300;
    const unsigned flag_sets[] = {0u,
                                  RESHARD_NO_GATHER,
                                  RESHARD_LDS_STAGING,
                                  RESHARD_NO_REALIGN | RESHARD_NO_GATHER,
                                  RESHARD_SENDER_NAIVE | RESHARD_TASK_ORDER,
                                  RESHARD_STRATEGY_SENDRECV,
                                  RESHARD_STRATEGY_ALLGATHER};
    const reshard_dtype_t dts[] = {RESHARD_U8, RESHARD_F16, RESHARD_F32, RESHARD_F64};
    const int64_t esz[] = {1, 2, 4, 8};
    int plans = 0;
    for (int it = 0; it < iters; ++it) {
        const int nd = 1 + int(rnd(4));
        int64_t shape[4];
        for (int d = 0; d < nd; ++d) shape[d] = rnd(8) == 0 ? 0 : int64_t(1 + rnd(40));
        const int di = int(rnd(4));
        const int smn = 1 + int(rnd(3)), dmn = 1 + int(rnd(3));
        int64_t sm[3], dm[3];
        for (int a = 0; a < smn; ++a) sm[a] = 1 + rnd(4);
        for (int a = 0; a < dmn; ++a) dm[a] = 1 + rnd(4);
        const std::string ss = random_spec(nd, smn), ds = random_spec(nd, dmn);
        for (unsigned flags : flag_sets) {
            reshard_tuning_t tn;
            std::memset(&tn, 0, sizeof(tn));
            tn.chunk_bytes = rnd(3) == 0 ? 0 : int64_t(16 + rnd(3000));
            tn.block_threads = 64 << rnd(5);
            tn.gather_band = int32_t(rnd(4));
            // permuted local layouts (not with the comparison strategies)
            int32_t sperm[4], dperm[4];
            for (int d = 0; d < nd; ++d) sperm[d] = dperm[d] = d;
            const bool permute = rnd(2) == 0 && !(flags & (RESHARD_STRATEGY_SENDRECV | RESHARD_STRATEGY_ALLGATHER));
            if (permute)
                for (int d = nd - 1; d > 0; --d) {
                    std::swap(sperm[d], sperm[rnd(uint32_t(d + 1))]);
                    std::swap(dperm[d], dperm[rnd(uint32_t(d + 1))]);
                }
            reshard_plan_t *p = nullptr;
            if (reshard_plan_permuted(nd, shape, dts[di], smn, sm, ss.c_str(), sperm, dmn, dm, ds.c_str(), dperm,
                                      flags, &tn, &p) != RESHARD_OK) {
                fprintf(stderr, "plan failed: %s\n", reshard_last_error());
                return 1;
            }
            ++plans;
            int64_t ns = 1, ndst = 1;
            for (int a = 0; a < smn; ++a) ns *= sm[a];
            for (int a = 0; a < dmn; ++a) ndst *= dm[a];
            std::vector<void *> sp(ns), dp(ndst);
            std::vector<int64_t> ls(nd);
            for (int64_t k = 0; k < ns; ++k) {
                reshard_plan_local_shape(p, 0, k, ls.data());
                int64_t n = esz[di];
                for (int d = 0; d < nd; ++d) n *= ls[d];
                sp[k] = n ? malloc(size_t(n)) : nullptr;
                if (n) memset(sp[k], int(k), size_t(n));
            }
            for (int64_t k = 0; k < ndst; ++k) {
                reshard_plan_local_shape(p, 1, k, ls.data());
                int64_t n = esz[di];
                for (int d = 0; d < nd; ++d) n *= ls[d];
                dp[k] = n ? malloc(size_t(n)) : nullptr;
            }
            if (reshard_debug_execute_host(p, sp.data(), dp.data()) != RESHARD_OK) {
                fprintf(stderr, "host execute failed: %s\n", reshard_last_error());
                return 1;
            }
            int64_t st[5];
            reshard_plan_stats(p, &st[0], &st[1], &st[2], &st[3], &st[4]);
            if (!(flags & (RESHARD_STRATEGY_SENDRECV | RESHARD_STRATEGY_ALLGATHER)) && st[2] > 0 && st[2] <= 64) {
                std::vector<int64_t> snd(static_cast<size_t>(st[2])), start(static_cast<size_t>(st[2]));
                int64_t span = 0, lb = 0, nodes = 0;
                for (int algo = 0; algo < 5; ++algo)
                    if (reshard_schedule(p, 1 + rnd(3), 1 + rnd(3), reshard_sched_algo_t(algo), 200, 4, rnd(1000),
                                         snd.data(), start.data(), &span, &lb, &nodes) != RESHARD_OK) {
                        fprintf(stderr, "schedule failed: %s\n", reshard_last_error());
                        return 1;
                    }
            }
            for (auto q : sp) free(q);
            for (auto q : dp) free(q);
            reshard_plan_destroy(p);
        }
    }
    // planning only, at sizes whose buffers would not fit this host: the two
    // innermost extents up to 2^16, tensors of 2^32 to 2^35 bytes, permuted
    // layouts included.
    // Each plan either builds with read and written bytes equal to the
    // definition (every element read once, every destination shard written
    // once) or fails with a clean status and message.
    for (int it = 0; it < iters / 10; ++it) {
        const int nd = 2 + int(rnd(3));
        const int di = int(rnd(4));
        int64_t shape[4], numel = 1;
        for (int d = 0; d < nd; ++d) {
            shape[d] = d + 2 >= nd ? int64_t(1 + rnd(1u << 16)) : int64_t(1 + rnd(16));
            numel *= shape[d];
        }
        if (numel * esz[di] < (int64_t(1) << 32) || numel * esz[di] > (int64_t(1) << 35)) {
            --it;
            continue;
        }
        const int smn = 1 + int(rnd(2)), dmn = 1 + int(rnd(2));
        int64_t sm[2], dm[2];
        for (int a = 0; a < smn; ++a) sm[a] = 1 + rnd(4);
        for (int a = 0; a < dmn; ++a) dm[a] = 1 + rnd(4);
        const std::string ss = random_spec(nd, smn), ds = random_spec(nd, dmn);
        int32_t sperm[4], dperm[4];
        for (int d = 0; d < nd; ++d) sperm[d] = dperm[d] = d;
        for (int d = nd - 1; d > 0; --d) {
            std::swap(sperm[d], sperm[rnd(uint32_t(d + 1))]);
            std::swap(dperm[d], dperm[rnd(uint32_t(d + 1))]);
        }
        reshard_plan_t *p = nullptr;
        const reshard_status_t st0 = reshard_plan_permuted(nd, shape, dts[di], smn, sm, ss.c_str(), sperm, dmn, dm,
                                                           ds.c_str(), dperm, 0u, nullptr, &p);
        if (st0 != RESHARD_OK) {
            const char *e = reshard_last_error();
            if (st0 != RESHARD_EUNSUPPORTED || !e || !*e) {
                fprintf(stderr, "big plan: status %d: %s\n", int(st0), e ? e : "(null)");
                return 1;
            }
            continue;
        }
        ++plans;
        int64_t st[5];
        reshard_plan_stats(p, &st[0], &st[1], &st[2], &st[3], &st[4]);
        int64_t ndst = 1, written = 0;
        for (int a = 0; a < dmn; ++a) ndst *= dm[a];
        std::vector<int64_t> ls(nd);
        for (int64_t k = 0; k < ndst; ++k) {
            reshard_plan_local_shape(p, 1, k, ls.data());
            int64_t n = esz[di];
            for (int d = 0; d < nd; ++d) n *= ls[d];
            written += n;
        }
        if (st[0] != numel * esz[di] || st[1] != written) {
            fprintf(stderr, "big plan: bytes %lld/%lld, want %lld/%lld\n", (long long)st[0], (long long)st[1],
                    (long long)(numel * esz[di]), (long long)written);
            return 1;
        }
        reshard_plan_destroy(p);
    }
    for (int S = 1; S <= 6; ++S)
        for (int M = 1; M <= 9; M += 4) {
            double lat = 0;
            std::vector<int32_t> peak(static_cast<size_t>(S));
            if (reshard_pipeline_simulate(S, M, S % 2, 1.0, 2.0, 0.5, 0.25, M % 2, &lat, peak.data()) != RESHARD_OK)
                return 1;
        }
    printf("ok %d\n", plans);
    return 0;
}
