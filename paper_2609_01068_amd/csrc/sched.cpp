// Control plane and decode-cluster simulation (Section 5, system-level
// evaluation: RR / least-predicted-work routing, FCFS / SJF queues).
#include "sched.hpp"

#include <cmath>

#include "outlets.h"

namespace outlets {

ControlPlane::ControlPlane(const SchedPolicy& p, int32_t capacity)
    : pol_(p), inst_(static_cast<size_t>(p.instances)), pred_(capacity, 0), gen_(capacity, 0),
      where_(capacity, -1), slot_(capacity, -1), state_(capacity, kIdle) {}

int ControlPlane::check_submit(int32_t n, const int32_t* ids, const int32_t* pred, const char** why) const {
    std::vector<char> seen;
    for (int32_t i = 0; i < n; ++i) {
        const int32_t id = ids[i];
        if (id < 0 || id >= capacity()) { *why = "request id out of range"; return OUTLETS_ERR_INVALID_ARG; }
        if (state_[id] != kIdle) { *why = "request id already waiting or running"; return OUTLETS_ERR_SLOT_BUSY; }
        if (pred[i] < 0) { *why = "predicted length must be >= 0"; return OUTLETS_ERR_INVALID_ARG; }
    }
    seen.assign(static_cast<size_t>(capacity()), 0);
    for (int32_t i = 0; i < n; ++i) {
        if (seen[ids[i]]) { *why = "repeated request id"; return OUTLETS_ERR_INVALID_ARG; }
        seen[ids[i]] = 1;
    }
    return OUTLETS_OK;
}

int32_t ControlPlane::submit(int32_t id, int32_t pred) {
    int32_t k = 0;
    if (pol_.routing == ROUTE_RR) {
        k = static_cast<int32_t>(submitted_ % pol_.instances);
    } else {
        for (int32_t j = 1; j < pol_.instances; ++j)
            if (inst_[j].load < inst_[k].load) k = j;
    }
    const int64_t key = (pol_.order == QUEUE_SJF) ? pred : 0;
    inst_[k].waiting.push({{key, submitted_}, id});
    inst_[k].load += pred;
    pred_[id] = pred;
    gen_[id] = 0;
    where_[id] = k;
    state_[id] = kWaiting;
    ++submitted_;
    return k;
}

int32_t ControlPlane::admit(int32_t k, int32_t cap, int32_t* out) {
    Instance& in = inst_[k];
    int32_t m = 0;
    while (m < cap && static_cast<int32_t>(in.running.size()) < pol_.max_running && !in.waiting.empty()) {
        const int32_t id = in.waiting.top().second;
        in.waiting.pop();
        state_[id] = kRunning;
        slot_[id] = static_cast<int32_t>(in.running.size());
        in.running.push_back(id);
        if (out) out[m] = id;
        ++m;
    }
    return m;
}

void ControlPlane::iteration(int32_t k) {
    Instance& in = inst_[k];
    for (int32_t id : in.running) {
        // remaining predicted work max(pred - gen, 0) drops while gen < pred
        if (gen_[id] < pred_[id]) in.load -= 1;
        gen_[id] += 1;
    }
}

void ControlPlane::finish(int32_t id) {
    Instance& in = inst_[where_[id]];
    if (gen_[id] < pred_[id]) in.load -= pred_[id] - gen_[id];
    const int32_t s = slot_[id];
    const int32_t last = in.running.back();
    in.running[s] = last;
    slot_[last] = s;
    in.running.pop_back();
    state_[id] = kIdle;
    slot_[id] = -1;
    where_[id] = -1;
}

int simulate(const SimConfig& cfg, int32_t n, const int64_t* arrival, const int32_t* out_len,
             const int32_t* pred, int32_t* instance_out, int64_t* start_out, int64_t* finish_out,
             const char** why) {
    const int32_t K = cfg.policy.instances;
    for (int32_t i = 0; i < n; ++i) {
        if (out_len[i] < 1) { *why = "true output lengths must be >= 1"; return OUTLETS_ERR_INVALID_ARG; }
        if (pred[i] < 0) { *why = "predicted lengths must be >= 0"; return OUTLETS_ERR_INVALID_ARG; }
        if (i > 0 && arrival[i] < arrival[i - 1]) { *why = "arrival times must be nondecreasing"; return OUTLETS_ERR_INVALID_ARG; }
    }
    ControlPlane cp(cfg.policy, n);
    std::vector<int64_t> iter_end(static_cast<size_t>(K), -1);   // -1: idle
    std::vector<int32_t> admitted(static_cast<size_t>(cfg.policy.max_running));
    int32_t next = 0, done = 0;
    while (done < n) {
        int64_t t = (next < n) ? arrival[next] : INT64_MAX;
        for (int32_t k = 0; k < K; ++k)
            if (iter_end[k] >= 0 && iter_end[k] < t) t = iter_end[k];
        // 1. iteration ends: one token per running request, then finishes
        for (int32_t k = 0; k < K; ++k) {
            if (iter_end[k] != t) continue;
            iter_end[k] = -1;
            cp.iteration(k);
            const std::vector<int32_t>& run = cp.running(k);
            for (int32_t j = static_cast<int32_t>(run.size()) - 1; j >= 0; --j) {
                const int32_t id = run[j];      // swap-removal only touches visited entries
                if (cp.generated(id) == out_len[id]) {
                    finish_out[id] = t;
                    cp.finish(id);
                    ++done;
                }
            }
        }
        // 2. arrivals, routed in arrival order
        for (; next < n && arrival[next] == t; ++next) instance_out[next] = cp.submit(next, pred[next]);
        // 3. admissions and iteration starts at idle instances
        for (int32_t k = 0; k < K; ++k) {
            if (iter_end[k] >= 0) continue;
            const int32_t m = cp.admit(k, cfg.policy.max_running, admitted.data());
            for (int32_t j = 0; j < m; ++j) start_out[admitted[j]] = t;
            const int64_t b = static_cast<int64_t>(cp.running(k).size());
            if (b > 0) iter_end[k] = t + cfg.iter_base_us + cfg.iter_per_seq_us * b;
        }
    }
    return OUTLETS_OK;
}

int32_t pred_tokens_from_z(float z) {
    if (z != z) return 0;
    const double r = std::fmax(0.0, std::expm1(static_cast<double>(z)));
    if (r >= 2147483646.5) return INT32_MAX;
    return static_cast<int32_t>(std::floor(r + 0.5));
}

}  // namespace outlets
