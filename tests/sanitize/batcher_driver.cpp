// Drives the host-side adaptive batcher through create, submit, step, probe,
// simulate and check on a seeded two-pipeline plan, under AddressSanitizer
// and UndefinedBehaviorSanitizer (test infrastructure).
#include "ppipe.h"

#include <cstdio>
#include <random>
#include <string>
#include <vector>

namespace ppipe {
int set_error(int status, const std::string&) { return status; }   // the runtime's error slot
}

int main()
{
    const int max_bs = 8;
    // pipeline 0: two stages on GPUs {0,1} and {2,3}; pipeline 1: one stage on {4,5}
    const int32_t n0[] = {2, 2}, g0[] = {0, 1, 2, 3};
    const int32_t n1[] = {2}, g1[] = {4, 5};
    std::vector<double> inf0(2 * max_bs), net0(2 * max_bs), inf1(max_bs), net1(max_bs, 0.0);
    for (int b = 1; b <= max_bs; ++b) {
        inf0[b - 1] = 300 + 40 * b;
        inf0[max_bs + b - 1] = 250 + 35 * b;
        net0[b - 1] = 0;
        net0[max_bs + b - 1] = 20 + 5 * b;
        inf1[b - 1] = 500 + 70 * b;
    }
    ppipe_pipeline_desc p[2] = {{2, n0, g0, max_bs, 4, inf0.data(), net0.data()},
                                {1, n1, g1, max_bs, 4, inf1.data(), net1.data()}};
    const int32_t node[] = {0, 0, 1, 1, 2, 2};
    ppipe_batcher* b = ppipe_batcher_create(6, node, 2, p);
    if (!b) return 2;
    // call by call
    ppipe_decision d;
    double fin = 0, wt = 0;
    int32_t path[PPIPE_MAX_STAGES];
    for (int i = 0; i < 20; ++i) ppipe_batcher_submit(b, i, 10.0 * i, 10.0 * i + 3000);
    for (int i = 0; i < 60; ++i) {
        if (ppipe_batcher_step(b, 200.0 + i, 0, &d) != 0) return 3;
        if (d.kind == PPIPE_DECISION_IDLE) break;
        if (d.kind == PPIPE_DECISION_WAIT && ppipe_batcher_step(b, d.wake_us, 1, &d) != 0) return 4;
    }
    ppipe_batcher_probe(b, 0, 3, 500.0, &fin, &wt, path);
    // event loop over seeded Poisson arrivals
    std::mt19937_64 rng(7);
    std::exponential_distribution<double> gap(1.0 / 60.0);
    std::vector<double> arr(5000);
    double t = 1e4;
    for (double& a : arr) a = (t += gap(rng));
    ppipe_sim_stats st{};
    std::vector<ppipe_decision> log(256);
    int64_t logged = 0;
    if (ppipe_batcher_simulate(b, arr.data(), (int64_t)arr.size(), 3000.0, &st, log.data(),
                               (int64_t)log.size(), &logged) != 0)
        return 5;
    int64_t overlaps = -1, intervals = 0;
    ppipe_batcher_check(b, &overlaps, &intervals);
    ppipe_batcher_destroy(b);
    std::printf("batcher sanitizer driver: %lld dispatched, %lld dropped, %lld overlaps\n",
                (long long)st.dispatched, (long long)st.dropped, (long long)overlaps);
    return overlaps == 0 && st.late == 0 ? 0 : 6;
}
