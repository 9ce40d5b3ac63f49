"""Oracle of the length-aware control plane that consumes the static
prediction r_hat_0 (Section 5, system-level evaluation in disaggregated
serving; appendix on the system evaluation).

TEST INFRASTRUCTURE ONLY (like the rest of ``oracle/``): plain Python lists
and loops, written from the paper's description of the two decisions, and
sharing no code with the C++ control plane.

Policies (Section 5 system setup):

* routing RR: request i (in arrival order) goes to decode instance i mod K;
* routing LB: a request goes to the instance with the lowest estimated
  remaining workload, the sum over its queued and running requests of their
  predicted remaining lengths; ties go to the lowest instance index;
* queue FCFS: an instance admits its waiting requests in arrival order;
* queue SJF: an instance admits the waiting request with the shortest
  predicted length first (ties in arrival order).

Readings where the paper gives no detail (stated again in the design notes):

* Predicted lengths are whole tokens: p = floor(max(0, expm1(z_hat)) + 0.5)
  from the length head's z_hat = log(1 + length) (Section 4.2).
* A running request's predicted remaining length is max(p - generated, 0);
  a queued request counts p.
* Service model: each decode instance runs continuous-batching iterations
  back to back while it has running requests.  At most S requests run at
  once; waiting requests are admitted only at an iteration boundary (or on
  arrival at an idle instance).  One iteration lasts base + per_seq * b
  microseconds for b running requests and gives every running request one
  token; a request finishes at the end of the iteration that produces its
  L-th token (L = its true output length).  Admission is non-preemptive.
* Events at the same instant are handled in this order: iteration ends (in
  instance order), then arrivals (in arrival order), then admissions and
  iteration starts at every idle instance (in instance order).
* Latency = finish - arrival; throughput = generated tokens / (last finish -
  first arrival); P99 is the nearest-rank percentile (the ceil(0.99 n)-th
  smallest); classes by true output length: short < 800, medium [800, 1300),
  long >= 1300 tokens (the appendix's table classes).
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

RR, LB = 0, 1
FCFS, SJF = 0, 1


def pred_tokens(z_hat: Sequence[float]) -> List[int]:
    """Whole-token predicted lengths from z_hat ~ log(1 + length) (Section
    4.2): floor(max(0, expm1(z)) + 0.5), capped at 2^31 - 1."""
    out = []
    for z in z_hat:
        z = float(z)
        r = 0.0 if z != z else max(0.0, math.expm1(z))       # NaN predicts 0
        out.append(2 ** 31 - 1 if r >= 2 ** 31 - 1.5 else int(math.floor(r + 0.5)))
    return out


def route(i: int, loads: List[int], routing: int) -> int:
    """Instance of the i-th arriving request: i mod K (RR) or the lowest
    estimated remaining work, lowest index on ties (LB)."""
    if routing == RR:
        return i % len(loads)
    return loads.index(min(loads))


def pick(waiting: List[int], pred: Sequence[int], order: int) -> int:
    """Next request to admit: earliest arrival (FCFS) or shortest predicted
    length, earliest arrival on ties (SJF)."""
    if order == FCFS:
        return min(waiting)
    return min(waiting, key=lambda i: (pred[i], i))


def finished(generated: int, length: int) -> bool:
    """A request is done once it has produced its true number of tokens."""
    return generated == length


def simulate(arrival: Sequence[int], out_len: Sequence[int], pred: Sequence[int], K: int, S: int,
             routing: int, order: int, base: int, per_seq: int) -> Tuple[List[int], List[int], List[int]]:
    """Serve the requests (arrival times in microseconds, nondecreasing) on K
    decode instances; returns per request (instance, start, finish)."""
    n = len(arrival)
    inst = [-1] * n
    start = [-1] * n
    finish = [-1] * n
    waiting = [[] for _ in range(K)]        # request ids
    running = [[] for _ in range(K)]        # request ids
    generated = [0] * n
    iter_end = [None] * K                   # end time of the iteration in progress
    nxt = 0                                 # next arrival to route

    def load(k):
        w = sum(pred[i] for i in waiting[k])
        return w + sum(max(pred[i] - generated[i], 0) for i in running[k])

    done = 0
    while done < n:
        times = [e for e in iter_end if e is not None]
        if nxt < n:
            times.append(arrival[nxt])
        t = min(times)
        # 1. iteration ends
        for k in range(K):
            if iter_end[k] == t:
                iter_end[k] = None
                still = []
                for i in running[k]:
                    generated[i] += 1
                    if finished(generated[i], out_len[i]):
                        finish[i] = t
                        done += 1
                    else:
                        still.append(i)
                running[k] = still
        # 2. arrivals
        while nxt < n and arrival[nxt] == t:
            i = nxt
            k = route(i, [load(k) for k in range(K)], routing)
            inst[i] = k
            waiting[k].append(i)
            nxt += 1
        # 3. admissions and iteration starts at idle instances
        for k in range(K):
            if iter_end[k] is not None:
                continue
            while len(running[k]) < S and waiting[k]:
                best = pick(waiting[k], pred, order)
                waiting[k].remove(best)
                running[k].append(best)
                start[best] = t
            if running[k]:
                iter_end[k] = t + base + per_seq * len(running[k])
    return inst, start, finish


def nearest_rank_p99(values: Sequence[float]) -> float:
    if not values:
        return float("nan")
    v = sorted(values)
    return v[(99 * len(v) + 99) // 100 - 1]       # rank ceil(0.99 n), in integers


def metrics(arrival, out_len, finish, short_below=800, long_from=1300):
    """(tokens/s, mean latency s, P99 short s, P99 medium s, P99 long s,
    makespan s) of one simulated run."""
    n = len(arrival)
    if n == 0:
        nan = float("nan")
        return (nan, nan, nan, nan, nan, nan)
    lat = [(finish[i] - arrival[i]) / 1e6 for i in range(n)]
    span = (max(finish) - min(arrival)) / 1e6
    short = [lat[i] for i in range(n) if out_len[i] < short_below]
    med = [lat[i] for i in range(n) if short_below <= out_len[i] < long_from]
    lng = [lat[i] for i in range(n) if out_len[i] >= long_from]
    tput = sum(out_len) / span if span > 0 else float("inf")
    return (tput, sum(lat) / n, nearest_rank_p99(short), nearest_rank_p99(med),
            nearest_rank_p99(lng), span)
