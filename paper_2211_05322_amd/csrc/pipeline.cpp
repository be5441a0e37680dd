// pipeline.cpp -- discrete-event model of the pipeline schedules of Section 4
// (1F1B and eager-1F1B) with cross-mesh resharding between stages.
//
// S stages, M micro-batches.  Stage s (0-based) runs its operations strictly
// in its schedule's order: w forwards, then alternately one backward and one
// forward, then the remaining backwards, where w = S - s for 1F1B (the paper
// counts #stages - i + 1 with stages from 1) and w = 2(S - s) - 1 for
// eager-1F1B (2(#stages - i) + 1), both capped at M.  F(s, m) needs F(s-1, m)
// and the transfer of its output from stage s-1; B(s, m) needs B(s+1, m) and
// the transfer of its gradient from stage s+1 (the last stage's backward
// follows its own forward).  A transfer starts when its producer finishes
// and, with `serial_links`, after the previous transfer on the same directed
// stage pair (a FIFO link); it takes the given communication time.
// Computation and communication overlap.  Reports the iteration latency and
// each stage's peak number of micro-batches whose forward is done and
// backward is not (live activations).
#include <algorithm>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/reshard.h"
#include "status.hpp"

extern "C" reshard_status_t reshard_pipeline_simulate(int32_t stages, int32_t microbatches, int32_t eager,
                                                      double t_fwd, double t_bwd, double t_comm_fwd,
                                                      double t_comm_bwd, int32_t serial_links,
                                                      double *latency_out, int32_t *peak_live_out) {
    return rs::guarded([&]() -> reshard_status_t {
        using rs::fail;
        const int S = stages, M = microbatches;
        if (S < 1 || M < 1 || S > 4096 || M > 1 << 20) return fail(RESHARD_EINVAL, "stages and micro-batches must be >= 1");
        if (t_fwd < 0 || t_bwd < 0 || t_comm_fwd < 0 || t_comm_bwd < 0) return fail(RESHARD_EINVAL, "negative time");
        // per-stage op lists: (is_backward, micro-batch)
        std::vector<std::vector<std::pair<int, int>>> ops(S);
        for (int s = 0; s < S; ++s) {
            int w = eager ? 2 * (S - s) - 1 : S - s;
            w = std::min(w, M);
            int nf = 0, nb = 0;
            for (; nf < w; ++nf) ops[s].push_back({0, nf});
            while (nf < M) {
                ops[s].push_back({1, nb++});
                ops[s].push_back({0, nf++});
            }
            while (nb < M) ops[s].push_back({1, nb++});
        }
        const double NA = -1.0;
        std::vector<std::vector<double>> f_done(S, std::vector<double>(M, NA)), b_done(S, std::vector<double>(M, NA));
        std::vector<std::vector<double>> f_arrive(S, std::vector<double>(M, NA)), b_arrive(S, std::vector<double>(M, NA));
        std::vector<double> link_fwd(S, 0.0), link_bwd(S, 0.0);  // link s: stage s -> s+1 / s+1 -> s
        std::vector<size_t> pos(S, 0);
        std::vector<double> stage_free(S, 0.0);
        std::vector<int> live(S, 0), peak(S, 0);
        size_t remaining = size_t(S) * size_t(M) * 2;
        double latency = 0.0;
        while (remaining) {
            // run every stage whose next op is ready, earliest start first
            int pick = -1;
            double pick_t = 0.0;
            for (int s = 0; s < S; ++s) {
                if (pos[s] == ops[s].size()) continue;
                const auto op = ops[s][pos[s]];
                double ready;
                if (op.first == 0) {
                    ready = s == 0 ? 0.0 : f_arrive[s][op.second];
                } else {
                    ready = s == S - 1 ? f_done[s][op.second] : b_arrive[s][op.second];
                }
                if (ready < 0) continue;  // producer not done yet
                const double t = std::max(stage_free[s], ready);
                if (pick < 0 || t < pick_t) {
                    pick = s;
                    pick_t = t;
                }
            }
            if (pick < 0) return fail(RESHARD_EINVAL, "internal: schedule deadlock");
            const int s = pick;
            const auto op = ops[s][pos[s]++];
            const int m = op.second;
            if (op.first == 0) {
                const double fin = pick_t + t_fwd;
                f_done[s][m] = fin;
                stage_free[s] = fin;
                peak[s] = std::max(peak[s], ++live[s]);
                if (s + 1 < S) {
                    const double st = serial_links ? std::max(fin, link_fwd[s]) : fin;
                    f_arrive[s + 1][m] = st + t_comm_fwd;
                    link_fwd[s] = st + t_comm_fwd;
                }
                latency = std::max(latency, fin);
            } else {
                const double fin = pick_t + t_bwd;
                b_done[s][m] = fin;
                stage_free[s] = fin;
                --live[s];
                if (s > 0) {
                    const double st = serial_links ? std::max(fin, link_bwd[s - 1]) : fin;
                    b_arrive[s - 1][m] = st + t_comm_bwd;
                    link_bwd[s - 1] = st + t_comm_bwd;
                }
                latency = std::max(latency, fin);
            }
            --remaining;
        }
        if (latency_out) *latency_out = latency;
        if (peak_live_out)
            for (int s = 0; s < S; ++s) peak_live_out[s] = peak[s];
        return RESHARD_OK;
    });
}
