"""The library's control plane (host C++) against the oracle, bit for bit:
the decode-cluster simulation, the whole-token prediction, the serving
metrics and the online submit / admit / iteration / finish calls (CPU only)."""
import json
import math
import os

import numpy as np
import pytest

import oracle.sched as S
from paper_2609_01068_amd import binding as B
from synth.serving import PAPER_TRACE, make_trace, noisy_predictions

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
POLICIES = [(S.RR, S.FCFS), (S.RR, S.SJF), (S.LB, S.FCFS), (S.LB, S.SJF)]


@pytest.fixture(scope="module", autouse=True)
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2609_01068_amd import build
        build.build(verbose=False)
    return B.lib()


def _both(a, L, p, K, Sl, routing, order, base, per):
    got = B.outlets_sched_simulate(a, L, p, K, Sl, routing, order, base, per)
    ref = S.simulate([int(x) for x in a], [int(x) for x in L], [int(x) for x in p], K, Sl, routing, order,
                     base, per)
    for g, r, what in zip(got, ref, ("instance", "start", "finish")):
        assert np.array_equal(g, np.asarray(r)), what
    return got


def test_hand_worked_example():
    with open(os.path.join(ROOT, "tests", "golden", "sched_example.json")) as f:
        ex = json.load(f)
    c, r = ex["cluster"], ex["requests"]
    names = {"RR+FCFS": POLICIES[0], "RR+SJF": POLICIES[1], "LB+FCFS": POLICIES[2], "LB+SJF": POLICIES[3]}
    for name, run in ex["runs"].items():
        got = B.outlets_sched_simulate(r["arrival_us"], r["out_len"], r["pred"], c["instances"],
                                       c["max_running"], *names[name], c["base_us"], c["per_seq_us"])
        assert [list(x) for x in got] == [run["instance"], run["start_us"], run["finish_us"]], name
    assert list(B.outlets_pred_tokens(ex["pred_tokens"]["z"])) == ex["pred_tokens"]["tokens"]


@pytest.mark.parametrize("K,Sl", [(1, 1), (2, 3), (3, 64), (5, 2)])
@pytest.mark.parametrize("policy", POLICIES, ids=["RR+FCFS", "RR+SJF", "LB+FCFS", "LB+SJF"])
def test_random_traces_match_oracle(K, Sl, policy):
    r = np.random.default_rng(K * 100 + Sl)
    for trial in range(6):
        n = int(r.integers(1, 300))
        # few distinct arrival instants and predictions: many ties
        a = np.sort(r.integers(0, 50, n) * int(r.integers(1, 40)))
        L = r.integers(1, 60, n)
        p = np.where(r.random(n) < 0.2, 0, r.integers(0, 30, n))
        base, per = [(5, 1), (0, 1), (1, 0), (40, 7), (0, 0)][trial % 5]
        _both(a, L, p, K, Sl, *policy, base, per)


@pytest.mark.parametrize("policy", POLICIES, ids=["RR+FCFS", "RR+SJF", "LB+FCFS", "LB+SJF"])
def test_paper_scale_trace_matches_oracle(policy):
    tr = PAPER_TRACE
    a, L = make_trace(tr)
    p = noisy_predictions(L, 0.25)
    _, _, fin = _both(a, L, p, tr.instances, tr.max_running, *policy, tr.iter_base_us, tr.iter_per_seq_us)
    got = B.outlets_sched_metrics(a, L, fin)
    ref = S.metrics([int(x) for x in a], [int(x) for x in L], [int(x) for x in fin])
    assert got[2:5] == ref[2:5] and got[5] == ref[5]
    assert got[0] == pytest.approx(ref[0], rel=1e-12) and got[1] == pytest.approx(ref[1], rel=1e-12)


def test_pred_tokens_match_oracle():
    r = np.random.default_rng(3)
    z = np.concatenate([r.normal(5, 3, 5000), [0.0, -0.0, -20.0, 30.0, np.nan, np.inf, -np.inf,
                                              np.log(1.5), np.log(2.5), 21.49]]).astype(np.float32)
    assert list(B.outlets_pred_tokens(z)) == S.pred_tokens(z)


def test_metrics_edge_cases():
    got = B.outlets_sched_metrics([5, 7], [900, 1000], [105, 7 + 10 ** 6])
    ref = S.metrics([5, 7], [900, 1000], [105, 7 + 10 ** 6])
    assert math.isnan(got[2]) and math.isnan(got[4]) and got[3] == ref[3]
    assert all(math.isnan(x) for x in B.outlets_sched_metrics([], [], []))


def test_empty_trace_and_input_errors():
    assert all(len(x) == 0 for x in B.outlets_sched_simulate([], [], [], 3, 4, 1, 1, 10, 1))
    bad = [([0, 5, 3], [1, 1, 1], [1, 1, 1]),      # arrivals not sorted
           ([0, 1, 2], [1, 0, 1], [1, 1, 1]),      # empty output
           ([0, 1, 2], [1, 1, 1], [1, -1, 1]),     # negative prediction
           ([-1, 1, 2], [1, 1, 1], [1, 1, 1])]     # negative time
    for a, L, p in bad:
        with pytest.raises(B.OutletsError) as e:
            B.outlets_sched_simulate(a, L, p, 2, 2, 1, 1, 10, 1)
        assert e.value.rc == B.OUTLETS_ERR_INVALID_ARG
    for K, Sl, rt, od, base in ((0, 1, 0, 0, 1), (1, 0, 0, 0, 1), (1, 1, 2, 0, 1), (1, 1, 0, 5, 1), (1, 1, 0, 0, -1)):
        with pytest.raises(B.OutletsError):
            B.outlets_sched_simulate([0], [1], [1], K, Sl, rt, od, base, 1)


def _drive_online(a, L, p, K, Sl, routing, order, base, per):
    """The decode-cluster event loop written over the online calls."""
    cp = B.ControlPlane(K, Sl, routing, order, len(a))
    n = len(a)
    inst, start, fin = [-1] * n, [-1] * n, [-1] * n
    gen = [0] * n
    running = [[] for _ in range(K)]
    end = [None] * K
    nxt = done = 0
    while done < n:
        t = min([e for e in end if e is not None] + ([int(a[nxt])] if nxt < n else []))
        for k in range(K):
            if end[k] == t:
                end[k] = None
                cp.iteration(k)
                fin_ids = []
                for i in running[k]:
                    gen[i] += 1
                    if gen[i] == L[i]:
                        fin_ids.append(i)
                        fin[i] = t
                if fin_ids:
                    cp.finish(fin_ids)
                    done += len(fin_ids)
                running[k] = [i for i in running[k] if gen[i] < L[i]]
        ids = []
        while nxt < n and a[nxt] == t:
            ids.append(nxt)
            nxt += 1
        for i in ids:        # one call per request so LB sees each routing
            inst[i] = cp.submit([i], [int(p[i])])[0]
        for k in range(K):
            if end[k] is None:
                for i in cp.admit(k):
                    start[i] = t
                    running[k].append(i)
                load, nw, nr = cp.read(k)
                assert nr == len(running[k])
                exp = sum(max(int(p[i]) - gen[i], 0) for i in running[k])
                assert load >= exp
                if running[k]:
                    end[k] = t + base + per * len(running[k])
    cp.close()
    return inst, start, fin


@pytest.mark.parametrize("policy", POLICIES, ids=["RR+FCFS", "RR+SJF", "LB+FCFS", "LB+SJF"])
def test_online_calls_reproduce_the_simulation(policy):
    r = np.random.default_rng(11)
    n = 150
    a = np.sort(r.integers(0, 400, n))
    L = r.integers(1, 30, n)
    p = r.integers(0, 40, n)
    got = _drive_online(a, L, p, 3, 4, *policy, 6, 2)
    ref = B.outlets_sched_simulate(a, L, p, 3, 4, *policy, 6, 2)
    for g, rr in zip(got, ref):
        assert np.array_equal(np.asarray(g), rr)


def test_online_loads_and_errors():
    cp = B.ControlPlane(2, 1, B.OUTLETS_ROUTE_LB, B.OUTLETS_QUEUE_SJF, 8)
    assert cp.submit([3, 5, 1], [10, 4, 3]) == [0, 1, 1]
    assert cp.read(0) == (10, 1, 0) and cp.read(1) == (7, 2, 0)
    assert cp.admit(1) == [1]                 # SJF: pred 3 before pred 4
    cp.iteration(1)
    cp.iteration(1)
    assert cp.read(1) == (4 + 1, 1, 1)        # running 3 - 2 = 1, waiting 4
    for _ in range(3):
        cp.iteration(1)                       # past its prediction: counts 0
    assert cp.read(1) == (4, 1, 1)
    for call, rc in ((lambda: cp.submit([5], [1]), B.OUTLETS_ERR_SLOT_BUSY),
                     (lambda: cp.submit([8], [1]), B.OUTLETS_ERR_INVALID_ARG),
                     (lambda: cp.submit([6, 6], [1, 1]), B.OUTLETS_ERR_INVALID_ARG),
                     (lambda: cp.submit([6], [-1]), B.OUTLETS_ERR_INVALID_ARG),
                     (lambda: cp.finish([5]), B.OUTLETS_ERR_INVALID_ARG),      # waiting, not running
                     (lambda: cp.admit(2), B.OUTLETS_ERR_INVALID_ARG),
                     (lambda: cp.iteration(-1), B.OUTLETS_ERR_INVALID_ARG)):
        with pytest.raises(B.OutletsError) as e:
            call()
        assert e.value.rc == rc
    assert cp.read(0) == (10, 1, 0) and cp.read(1) == (4, 1, 1)   # failed calls changed nothing
    cp.finish([1])
    assert cp.read(1) == (4, 1, 0)
    assert cp.submit([1], [2]) == [1]         # a finished id can be reused
    cp.close()
