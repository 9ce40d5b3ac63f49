// Length-aware control plane of the disaggregated serving experiment
// (Section 5, system-level evaluation): routing of arriving requests over
// decode instances (round-robin, or least predicted remaining work) and the
// admission order of each instance's queue (arrival order, or shortest
// predicted length first), driven by the static length prediction.
// Host code only.
#pragma once

#include <cstdint>
#include <queue>
#include <utility>
#include <vector>

namespace outlets {

enum { ROUTE_RR = 0, ROUTE_LB = 1 };
enum { QUEUE_FCFS = 0, QUEUE_SJF = 1 };

struct SchedPolicy {
    int32_t instances = 1;    // decode instances K
    int32_t max_running = 1;  // concurrently running requests per instance S
    int32_t routing = ROUTE_RR;
    int32_t order = QUEUE_FCFS;
};

// Per-request state lives in flat arrays indexed by the caller's request id
// in [0, capacity).  Loads are whole predicted tokens, kept exactly.
class ControlPlane {
public:
    ControlPlane(const SchedPolicy& p, int32_t capacity);

    int32_t capacity() const { return static_cast<int32_t>(pred_.size()); }
    int32_t instances() const { return pol_.instances; }

    // Checks (no state change): id range, idle ids, no repeats, pred >= 0.
    int check_submit(int32_t n, const int32_t* ids, const int32_t* pred, const char** why) const;
    // Route and enqueue one checked request; returns its instance.
    int32_t submit(int32_t id, int32_t pred);
    // Move up to min(cap, S - running) waiting requests of instance k to
    // running, best first; writes their ids to out and returns the count.
    int32_t admit(int32_t k, int32_t cap, int32_t* out);
    // One decode iteration of instance k: every running request gains a token.
    void iteration(int32_t k);
    // End a running request.
    void finish(int32_t id);

    bool is_running(int32_t id) const { return state_[id] == kRunning; }
    int32_t generated(int32_t id) const { return gen_[id]; }
    const std::vector<int32_t>& running(int32_t k) const { return inst_[k].running; }
    int64_t load(int32_t k) const { return inst_[k].load; }
    int32_t n_waiting(int32_t k) const { return static_cast<int32_t>(inst_[k].waiting.size()); }

private:
    enum : int8_t { kIdle = 0, kWaiting = 1, kRunning = 2 };
    // (priority key, submission sequence, id); smallest first
    using Entry = std::pair<std::pair<int64_t, int64_t>, int32_t>;
    struct Instance {
        std::priority_queue<Entry, std::vector<Entry>, std::greater<Entry>> waiting;
        std::vector<int32_t> running;
        int64_t load = 0;     // predicted remaining tokens of waiting + running
    };
    SchedPolicy pol_;
    std::vector<Instance> inst_;
    std::vector<int32_t> pred_, gen_, where_, slot_;
    std::vector<int8_t> state_;
    int64_t submitted_ = 0;
};

struct SimConfig {
    SchedPolicy policy;
    int64_t iter_base_us = 0;     // iteration time = base + per_seq * running
    int64_t iter_per_seq_us = 0;
};

// Discrete-event run of the decode cluster over a request trace (arrival
// times nondecreasing, true lengths >= 1, predictions >= 0).
int simulate(const SimConfig& cfg, int32_t n, const int64_t* arrival, const int32_t* out_len,
             const int32_t* pred, int32_t* instance_out, int64_t* start_out, int64_t* finish_out,
             const char** why);

// Whole-token prediction from z_hat = log(1 + length): floor(max(0, expm1 z)
// + 0.5), NaN -> 0, capped at 2^31 - 1.
int32_t pred_tokens_from_z(float z);

}  // namespace outlets
