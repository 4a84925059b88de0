// Resource-reservation adaptive batching (Sec. 5.4; Alg. 1 and Alg. 2 of the
// appendix), host only.  The operations and their contracts are stated with
// the declarations in ppipe.h; this file keeps the reservation tables and
// makes the decisions without allocating on the probe path.
#include "ppipe.h"

#include <algorithm>
#include <chrono>
#include <cmath>
#include <deque>
#include <limits>
#include <memory>
#include <string>
#include <vector>

namespace ppipe {
int set_error(int status, const std::string& msg);   // runtime.hip
}

namespace {

constexpr double INF = std::numeric_limits<double>::infinity();

struct Interval {
    double start, end;   // half-open [start, end), end > start
};

// Reserved intervals of one resource, sorted and disjoint, so their ends
// increase too and the one interval that can block a slot starting at t is
// the first that ends after t.  `head` skips the intervals that ended by
// `past` (the latest decision time seen): a search from t >= past starts
// there, which keeps it to the few reservations still ahead.
struct Resource {
    std::vector<Interval> busy;
    size_t head = 0;

    const Interval* first_ending_after(double t, double past)
    {
        while (head < busy.size() && busy[head].end <= past) ++head;
        auto from = busy.begin() + (t >= past ? (std::ptrdiff_t)head : 0);
        auto it = std::upper_bound(from, busy.end(), t,
                                   [](double v, const Interval& iv) { return v < iv.end; });
        return it == busy.end() ? nullptr : &*it;
    }
    void mark(double start, double dur)
    {
        if (!(dur > 0)) return;   // an empty interval occupies nothing
        auto it = std::upper_bound(busy.begin(), busy.end(), start,
                                   [](double v, const Interval& x) { return v < x.start; });
        // an interval placed before an ended one has ended too
        if ((size_t)(it - busy.begin()) < head) ++head;
        busy.insert(it, Interval{start, start + dur});
    }
};

struct Stage {
    std::vector<int> gpus;
    std::vector<double> infer, net;   // [bs - 1]
};

struct Pipeline {
    std::vector<Stage> stages;
    int bs = 1, max_bs = 1;
};

struct Resv {
    int res;
    double start, dur;
};

// Outcome of a probe: at most a transfer (two links) and an inference per stage.
struct Probe {
    int n_stages = 0, n_resv = 0;
    int path[PPIPE_MAX_STAGES];
    Resv resv[3 * PPIPE_MAX_STAGES];
    double finish = INF, wait = 0;
};

struct Request {
    int64_t id;
    double arrival, deadline;
};

}  // namespace

struct ppipe_batcher {
    int n_gpus = 0, n_nodes = 0;
    std::vector<int> node;        // node of each GPU
    std::vector<Resource> res;    // GPUs, then node uplinks, then node downlinks
    std::vector<Pipeline> pipes;
    std::deque<Request> q;
    int64_t probes = 0;
    double past = -INF;   // latest time a decision or probe was made at

    int ul_res(int g) const { return n_gpus + node[g]; }
    int dl_res(int g) const { return n_gpus + n_nodes + node[g]; }

    // earliest time >= t at which every resource of rs is free for l:
    // push the candidate past every interval that blocks it until none does
    double earliest_slot(const int* rs, int n, double t, double l)
    {
        double tau = t;
        for (bool moved = true; moved;) {
            moved = false;
            for (int k = 0; k < n; ++k) {
                const Interval* iv = res[rs[k]].first_ending_after(tau, past);
                if (iv && iv->start < tau + l) {
                    tau = iv->end;
                    moved = true;
                }
            }
        }
        return tau;
    }

    void probe(int p, int bs, double now, Probe& out)
    {
        ++probes;
        past = std::max(past, now);
        const Pipeline& pl = pipes[p];
        out.n_stages = (int)pl.stages.size();
        out.n_resv = 0;
        out.wait = 0;
        double tg = now;
        int last = -1;
        for (int s = 0; s < out.n_stages; ++s) {
            const Stage& st = pl.stages[s];
            const double ln = st.net[bs - 1], li = st.infer[bs - 1];
            double best_t = INF, best_w = 0;
            int best_g = -1, best_n = 0;
            Resv best_r[3], r[3];
            for (int g : st.gpus) {
                double t = tg, w = 0;
                int n = 0;
                if (s > 0) {
                    const int links[2] = {ul_res(last), dl_res(g)};
                    const double tau = earliest_slot(links, 2, t, ln);
                    r[n++] = {links[0], tau, ln};
                    r[n++] = {links[1], tau, ln};
                    w += tau - t;
                    t = tau + ln;
                }
                const double tau = earliest_slot(&g, 1, t, li);
                r[n++] = {g, tau, li};
                w += tau - t;
                t = tau + li;
                if (t < best_t) {
                    best_t = t;
                    best_w = w;
                    best_g = g;
                    best_n = n;
                    std::copy(r, r + n, best_r);
                }
            }
            tg = best_t;
            last = best_g;
            out.path[s] = best_g;
            std::copy(best_r, best_r + best_n, out.resv + out.n_resv);
            out.n_resv += best_n;
            out.wait += best_w;
        }
        out.finish = tg;
    }

    void reserve(const Probe& r)
    {
        for (int k = 0; k < r.n_resv; ++k) res[r.resv[k].res].mark(r.resv[k].start, r.resv[k].dur);
    }

    void step(double now, bool deadline_wake, ppipe_decision* d)
    {
        *d = ppipe_decision{};
        d->pipeline = -1;
        d->wake_us = INF;
        for (int s = 0; s < PPIPE_MAX_STAGES; ++s) d->path[s] = -1;
        if (q.empty()) {
            d->kind = PPIPE_DECISION_IDLE;
            return;
        }
        const int64_t p0 = probes;
        // step 1: the pipeline that waits least at its unified batch size
        Probe cand, chosen;
        int best = -1;
        double best_wait = INF;
        for (int p = 0; p < (int)pipes.size(); ++p) {
            probe(p, pipes[p].bs, now, cand);
            if (cand.wait < best_wait) {
                best_wait = cand.wait;
                best = p;
                chosen = cand;
            }
        }
        // step 2: the largest batch from there down that meets the oldest
        // deadline (the step-1 probe already is the first candidate)
        const Pipeline& pl = pipes[best];
        const double deadline = q.front().deadline;
        const int cap = deadline_wake ? std::min<int>(pl.bs, (int)q.size()) : pl.bs;
        int bs_star = 0;
        for (int bs = cap; bs >= 1; --bs) {
            if (bs != pl.bs) probe(best, bs, now, chosen);
            if (chosen.finish <= deadline) {
                bs_star = bs;
                break;
            }
        }
        d->pipeline = best;
        if (bs_star == 0) {
            d->kind = PPIPE_DECISION_DROP;
            d->bs = 1;
            d->first_id = q.front().id;
            q.pop_front();
        } else if ((int)q.size() < bs_star) {
            // the queued requests can still start as late as their slack allows
            probe(best, (int)q.size(), now, cand);
            d->kind = PPIPE_DECISION_WAIT;
            d->bs = bs_star;
            d->wake_us = now + std::max(0.0, deadline - cand.finish);
        } else {
            reserve(chosen);
            d->kind = PPIPE_DECISION_DISPATCH;
            d->bs = bs_star;
            d->first_id = q.front().id;
            d->start_us = chosen.resv[0].start;
            d->finish_us = chosen.finish;
            d->deadline_us = deadline;
            std::copy(chosen.path, chosen.path + chosen.n_stages, d->path);
            q.erase(q.begin(), q.begin() + bs_star);
        }
        d->probes = (int32_t)(probes - p0);
    }
};

namespace {

ppipe_batcher* build(int32_t n_gpus, const int32_t* gpu_node, int32_t n_pipelines,
                     const ppipe_pipeline_desc* pipelines, std::string& err)
{
    if (n_gpus < 1 || n_pipelines < 1 || !pipelines) {
        err = "need at least one GPU and one pipeline";
        return nullptr;
    }
    std::unique_ptr<ppipe_batcher> b(new ppipe_batcher);
    b->n_gpus = n_gpus;
    b->node.resize(n_gpus);
    for (int g = 0; g < n_gpus; ++g) {
        b->node[g] = gpu_node ? gpu_node[g] : g;
        if (b->node[g] < 0 || b->node[g] >= n_gpus) {
            err = "GPU " + std::to_string(g) + ": node index outside [0, n_gpus)";
            return nullptr;
        }
        b->n_nodes = std::max(b->n_nodes, b->node[g] + 1);
    }
    b->res.resize((size_t)n_gpus + 2 * (size_t)b->n_nodes);
    for (int p = 0; p < n_pipelines; ++p) {
        const ppipe_pipeline_desc& d = pipelines[p];
        const std::string who = "pipeline " + std::to_string(p) + ": ";
        if (d.n_stages < 1 || d.n_stages > PPIPE_MAX_STAGES || !d.stage_n_gpus || !d.stage_gpus ||
            !d.infer_us || !d.net_us || d.max_bs < 1 || d.unified_bs < 1 ||
            d.unified_bs > d.max_bs) {
            err = who + "bad stage count, table pointer or batch size";
            return nullptr;
        }
        Pipeline pl;
        pl.bs = d.unified_bs;
        pl.max_bs = d.max_bs;
        size_t off = 0;
        for (int s = 0; s < d.n_stages; ++s) {
            Stage st;
            if (d.stage_n_gpus[s] < 1) {
                err = who + "stage " + std::to_string(s) + " has no GPU";
                return nullptr;
            }
            for (int k = 0; k < d.stage_n_gpus[s]; ++k) {
                const int g = d.stage_gpus[off++];
                if (g < 0 || g >= n_gpus) {
                    err = who + "GPU id " + std::to_string(g) + " out of range";
                    return nullptr;
                }
                st.gpus.push_back(g);
            }
            const double* inf = d.infer_us + (size_t)s * d.max_bs;
            const double* net = d.net_us + (size_t)s * d.max_bs;
            st.infer.assign(inf, inf + d.max_bs);
            st.net.assign(net, net + d.max_bs);
            for (int i = 0; i < d.max_bs; ++i)
                if (!(st.infer[i] >= 0 && st.infer[i] < INF) || !(st.net[i] >= 0 && st.net[i] < INF)) {
                    err = who + "latencies must be finite and >= 0";
                    return nullptr;
                }
            pl.stages.push_back(std::move(st));
        }
        b->pipes.push_back(std::move(pl));
    }
    return b.release();
}

}  // namespace

extern "C" {

ppipe_batcher* ppipe_batcher_create(int32_t n_gpus, const int32_t* gpu_node,
                                    int32_t n_pipelines, const ppipe_pipeline_desc* pipelines)
{
    std::string err;
    ppipe_batcher* b = build(n_gpus, gpu_node, n_pipelines, pipelines, err);
    if (!b) ppipe::set_error(PPIPE_E_INVALID, err);
    return b;
}

void ppipe_batcher_destroy(ppipe_batcher* b) { delete b; }

int ppipe_batcher_submit(ppipe_batcher* b, int64_t id, double arrival_us, double deadline_us)
{
    if (!b) return ppipe::set_error(PPIPE_E_INVALID, "null batcher");
    if (!std::isfinite(arrival_us) || !std::isfinite(deadline_us))
        return ppipe::set_error(PPIPE_E_INVALID, "arrival and deadline must be finite");
    if (!b->q.empty() && arrival_us < b->q.back().arrival)
        return ppipe::set_error(PPIPE_E_INVALID, "requests must be submitted in arrival order");
    b->q.push_back({id, arrival_us, deadline_us});
    return PPIPE_OK;
}

int ppipe_batcher_step(ppipe_batcher* b, double now_us, int32_t deadline_wake, ppipe_decision* d)
{
    if (!b || !d) return ppipe::set_error(PPIPE_E_INVALID, "null argument");
    if (!std::isfinite(now_us)) return ppipe::set_error(PPIPE_E_INVALID, "now must be finite");
    b->step(now_us, deadline_wake != 0, d);
    return PPIPE_OK;
}

int ppipe_batcher_probe(ppipe_batcher* b, int32_t pipeline, int32_t bs, double now_us,
                        double* finish_us, double* wait_us, int32_t* path)
{
    if (!b || pipeline < 0 || pipeline >= (int)b->pipes.size() || bs < 1 ||
        bs > b->pipes[pipeline].max_bs || !std::isfinite(now_us))
        return ppipe::set_error(PPIPE_E_INVALID, "bad batcher, pipeline, batch size or time");
    Probe r;
    b->probe(pipeline, bs, now_us, r);
    if (finish_us) *finish_us = r.finish;
    if (wait_us) *wait_us = r.wait;
    if (path) std::copy(r.path, r.path + r.n_stages, path);
    return PPIPE_OK;
}

int ppipe_batcher_check(const ppipe_batcher* b, int64_t* overlaps, int64_t* intervals)
{
    if (!b || !overlaps || !intervals) return ppipe::set_error(PPIPE_E_INVALID, "null argument");
    *overlaps = 0;
    *intervals = 0;
    for (const Resource& r : b->res) {
        *intervals += (int64_t)r.busy.size();
        for (size_t i = 1; i < r.busy.size(); ++i)
            if (r.busy[i].start < r.busy[i - 1].end) ++*overlaps;
    }
    return PPIPE_OK;
}

int ppipe_batcher_simulate(ppipe_batcher* b, const double* arrivals_us, int64_t n, double slo_us,
                           ppipe_sim_stats* stats, ppipe_decision* log, int64_t log_capacity,
                           int64_t* log_count)
{
    if (!b || (!arrivals_us && n > 0) || n < 0 || !stats || !(slo_us > 0) || !(slo_us < INF) ||
        (log_capacity > 0 && !log))
        return ppipe::set_error(PPIPE_E_INVALID, "bad simulation arguments");
    for (int64_t i = 0; i < n; ++i)
        if (!std::isfinite(arrivals_us[i]) || (i > 0 && arrivals_us[i] < arrivals_us[i - 1]))
            return ppipe::set_error(PPIPE_E_INVALID, "arrivals must be finite and sorted");
    if (!b->q.empty() && n > 0 && arrivals_us[0] < b->q.back().arrival)
        return ppipe::set_error(PPIPE_E_INVALID, "arrivals precede queued requests");
    *stats = ppipe_sim_stats{};
    using clock = std::chrono::steady_clock;
    int64_t logged = 0, next = 0;
    double wake = INF;
    while (next < n || !b->q.empty()) {
        const double ta = next < n ? arrivals_us[next] : INF;
        double now;
        bool at_wake;
        if (ta <= wake) {   // an arrival first (one at the wake time too)
            now = ta;
            at_wake = false;
            b->q.push_back({next, ta, ta + slo_us});
            ++next;
            ++stats->requests;
        } else {
            now = wake;
            at_wake = true;
        }
        wake = INF;
        for (;;) {
            ppipe_decision d;
            const auto t0 = clock::now();
            b->step(now, at_wake, &d);
            const double us = std::chrono::duration<double, std::micro>(clock::now() - t0).count();
            stats->decision_us += us;
            ++stats->decisions;
            stats->probes += d.probes;
            at_wake = false;   // only the first decision of a wake-up is forced
            if (d.kind != PPIPE_DECISION_IDLE && logged < log_capacity) log[logged++] = d;
            if (d.kind == PPIPE_DECISION_DISPATCH) {
                ++stats->batches;
                stats->dispatch_us += us;
                stats->dispatch_probes += d.probes;
                stats->dispatched += d.bs;
                if (d.finish_us > d.deadline_us) stats->late += d.bs;
                stats->max_finish_us = std::max(stats->max_finish_us, d.finish_us);
            } else if (d.kind == PPIPE_DECISION_DROP) {
                ++stats->dropped;
            } else {
                if (d.kind == PPIPE_DECISION_WAIT) wake = d.wake_us;
                break;
            }
        }
    }
    if (log_count) *log_count = logged;
    return PPIPE_OK;
}

}  // extern "C"
