"""Pins of the control-plane oracle (Section 5 system evaluation: RR / LB
routing, FCFS / SJF queues) against a hand-worked trace, closed forms of
the service model and textbook scheduling facts (CPU only)."""
import json
import os

import numpy as np
import pytest

import oracle.sched as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
POLICIES = {"RR+FCFS": (S.RR, S.FCFS), "RR+SJF": (S.RR, S.SJF), "LB+FCFS": (S.LB, S.FCFS),
            "LB+SJF": (S.LB, S.SJF)}


def _example():
    with open(os.path.join(ROOT, "tests", "golden", "sched_example.json")) as f:
        return json.load(f)


def _check_golden():
    ex = _example()
    c, r = ex["cluster"], ex["requests"]
    for name, run in ex["runs"].items():
        out = S.simulate(r["arrival_us"], r["out_len"], r["pred"], c["instances"], c["max_running"],
                         *POLICIES[name], c["base_us"], c["per_seq_us"])
        assert list(out) == [run["instance"], run["start_us"], run["finish_us"]], name


def test_hand_worked_example():
    _check_golden()


def test_pred_tokens_hand_values():
    ex = _example()["pred_tokens"]
    assert S.pred_tokens(ex["z"]) == ex["tokens"]
    assert S.pred_tokens([float("nan"), float("inf"), float("-inf"), 30.0]) == [0, 2 ** 31 - 1, 0, 2 ** 31 - 1]


def _trace(n, seed, t_max=2000, l_max=40):
    r = np.random.default_rng(seed)
    a = np.sort(r.integers(0, t_max, n))
    L = r.integers(1, l_max, n)
    p = np.maximum(0, L + r.integers(-10, 10, n))
    return [int(x) for x in a], [int(x) for x in L], [int(x) for x in p]


def _check_single_slot_fcfs_closed_form():
    # one instance, one slot, FCFS: requests are served back to back, each
    # taking L iterations of base + per_seq
    a, L, p = _trace(40, 1)
    base, per = 7, 3
    inst, start, fin = S.simulate(a, L, p, 1, 1, S.RR, S.FCFS, base, per)
    prev = 0
    for i in range(len(a)):
        s = max(a[i], prev)
        assert start[i] == s and fin[i] == s + L[i] * (base + per), i
        prev = fin[i]
    assert inst == [0] * len(a)


def test_single_slot_fcfs_is_a_sequential_queue():
    _check_single_slot_fcfs_closed_form()


def _check_unit_iterations_without_queueing():
    # enough slots and 1 us iterations: nobody waits, finish = arrival + L
    for (routing, order) in POLICIES.values():
        for K in (1, 3):
            a, L, p = _trace(60, 2 + K)
            inst, start, fin = S.simulate(a, L, p, K, 1000, routing, order, 1, 0)
            assert start == a
            assert fin == [a[i] + L[i] for i in range(len(a))]


def test_unit_iterations_without_queueing_finish_at_arrival_plus_length():
    _check_unit_iterations_without_queueing()


def _check_sjf_batch_order():
    # all requests present at t = 0 on one single-slot instance: SJF serves in
    # (pred, index) order; with exact predictions it minimises the mean
    # completion time (shortest processing time first), never above FCFS
    r = np.random.default_rng(5)
    L = [int(x) for x in r.integers(1, 50, 30)]
    L[3] = L[7]                                       # a tie, served in index order
    a = [0] * len(L)
    _, start, fin = S.simulate(a, L, L, 1, 1, S.RR, S.SJF, 2, 1)
    order = sorted(range(len(L)), key=lambda i: (L[i], i))
    t = 0
    for i in order:
        assert start[i] == t
        t += 3 * L[i]
        assert fin[i] == t
    _, _, fin_fcfs = S.simulate(a, L, L, 1, 1, S.RR, S.FCFS, 2, 1)
    assert sum(fin) <= sum(fin_fcfs)


def test_sjf_serves_a_batch_shortest_first_and_minimises_mean_completion():
    _check_sjf_batch_order()


def test_round_robin_assignment():
    a, L, p = _trace(50, 6)
    for order in (S.FCFS, S.SJF):
        inst, _, _ = S.simulate(a, L, p, 4, 2, S.RR, order, 5, 1)
        assert inst == [i % 4 for i in range(50)]


def _check_lb_greedy_bound():
    # simultaneous arrivals are all routed before any admission; greedy
    # least-loaded assignment keeps the loads within one job of each other
    r = np.random.default_rng(8)
    for K in (2, 3, 5):
        p = [int(x) for x in r.integers(0, 100, 40)]
        L = [1] * 40
        inst, _, _ = S.simulate([0] * 40, L, p, K, 4, S.LB, S.SJF, 5, 1)
        loads = [sum(p[i] for i in range(40) if inst[i] == k) for k in range(K)]
        assert max(loads) - min(loads) <= max(p)
        assert inst[0] == 0


def test_least_loaded_routing_balances_simultaneous_arrivals():
    _check_lb_greedy_bound()


def test_lb_counts_running_work_as_predicted_remaining():
    # instance 0 runs a request predicted at 10 tokens; after 4 iterations its
    # remaining estimate is 6, so a request arriving then (pred 7) goes to
    # instance 1 only if 1's load is below 6
    a = [0, 0, 40]
    L = [10, 20, 3]
    p = [10, 5, 7]
    inst, _, _ = S.simulate(a, L, p, 2, 4, S.LB, S.FCFS, 9, 1)     # 10 us per single-request iteration
    # at t = 40: instance 0 remaining 10 - 4 = 6, instance 1 remaining 5 - 4 = 1
    assert inst == [0, 1, 1]
    p2 = [10, 12, 7]
    inst2, _, _ = S.simulate(a, L, p2, 2, 4, S.LB, S.FCFS, 9, 1)
    # instance 1 remaining 12 - 4 = 8 > 6
    assert inst2 == [0, 1, 0]


def test_metrics_hand_values():
    arrival = [0, 1_000_000, 2_000_000, 2_000_000]
    out_len = [100, 900, 1500, 10]
    finish = [3_000_000, 4_000_000, 9_000_000, 2_500_000]
    tput, mean, p_s, p_m, p_l, span = S.metrics(arrival, out_len, finish)
    assert span == 9.0 and tput == 2510 / 9.0
    assert mean == (3.0 + 3.0 + 7.0 + 0.5) / 4
    assert (p_s, p_m, p_l) == (3.0, 3.0, 7.0)      # nearest rank of {3, 0.5} is its max
    assert S.nearest_rank_p99(list(range(1, 201))) == 198
    assert S.nearest_rank_p99(list(range(1, 101))) == 99


# ------------------------------------------------------------- planted mistakes

def _fails(fn):
    try:
        fn()
    except AssertionError:
        return True
    return False


def test_planted_argmax_routing_is_caught(monkeypatch):
    real = S.route
    monkeypatch.setattr(S, "route", lambda i, loads, r: real(i, loads, r) if r == S.RR
                        else loads.index(max(loads)))
    assert _fails(_check_golden) and _fails(_check_lb_greedy_bound)


def test_planted_longest_first_queue_is_caught(monkeypatch):
    real = S.pick
    monkeypatch.setattr(S, "pick", lambda w, p, o: real(w, p, o) if o == S.FCFS
                        else min(w, key=lambda i: (-p[i], i)))
    assert _fails(_check_golden) and _fails(_check_sjf_batch_order)


def test_planted_off_by_one_token_count_is_caught(monkeypatch):
    monkeypatch.setattr(S, "finished", lambda g, L: g == L + 1)
    assert _fails(_check_golden) and _fails(_check_unit_iterations_without_queueing)
    assert _fails(_check_single_slot_fcfs_closed_form)
