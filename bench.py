"""Throughput of the OUTLETS length-prediction hot path on one MI355X.

A step is one pass of the whole path over one batch: a static prediction for
every request of the batch (outlets_predict_prefill: fused projection, draft
layer, pooling, length head, paged KV write), one dynamic re-prediction per
request (outlets_predict_step: one new token per request through the same
layer against the paged KV cache), and the release of the requests' slots.

Default workload: the 8B-shaped bf16 draft layer (d 4096, 32 q / 8 KV heads,
head_dim 128, SwiGLU 14336, head 8192 -> 1024 -> 1) over 32 requests with
lognormal(median 512, sigma 1.0) prompt lengths clipped to [32, 4096],
synthetic seeded inputs resident in HBM before timing.  The same line
carries, under ``decode_step``, the decode-step half of the metric on the
HBM-bound per-step workload (512 in-flight requests with paged draft KV
caches of U[256, 8192] tokens): ms per step, draft tokens/s, and the
attention kernel's and the whole step's fraction of the HBM peak.

Prints one JSON line (rank 0).  ``--gpus`` above 1 is refused: the
benchmark measures one GPU's share of the request-parallel path.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "predicted requests/sec + draft tokens/sec at 8B shape; MFMA util / HBM GB/s"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0      # MI355X dense fp8 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E


def gemm_flops(shape, T: int, attn_gate: bool = False, input_embed: bool = False):
    """Algorithmic FLOPs per launch of each GEMM group for T tokens (the QKV
    GEMM also produces the Gated Attention gate when ``attn_gate``, and reads
    2d columns with input embeddings)."""
    d, hd = shape.d, shape.head_dim
    qkv = (shape.n_q * (2 if attn_gate else 1) + 2 * shape.n_kv) * hd
    return {
        "FUSE_GEMM": 2.0 * T * d * 3 * d,
        "QKV_GEMM": 2.0 * T * qkv * d * (2 if input_embed else 1),
        "O_GEMM": 2.0 * T * d * shape.n_q * hd,
        "GATE_UP_GEMM": 2.0 * T * 2 * shape.ffn * d,
        "DOWN_GEMM": 2.0 * T * d * shape.ffn,
    }


def recorded_traffic(profile="gate_up_gemm_8b_prefill_b32.md", source="gemm.hip", key="gemm"):
    """HBM bytes per launch of a dominant kernel from its committed rocprofv3
    counter summary, or None when the kernel's source file has changed since
    the counters were taken."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", profile)
    src = os.path.join(ROOT, "paper_2609_01068_amd", "csrc", source)
    try:
        text = open(path).read()
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    except OSError:
        return None
    vals = dict(re.findall(r"^(\w+): (\S+)$", text, re.M))
    if vals.get(f"{key}_source_sha256_16") != sha or "traffic_bytes_per_launch" not in vals:
        return None
    return float(vals["traffic_bytes_per_launch"])


def cpu_baseline(wl, W, lens, budget_s: float = 12.0):
    """The fp64 oracle on a bounded sample of the same batch: requests in
    batch order, static prediction + one step each, until ``budget_s`` of
    work; scaled to requests/s of the batch's mean request length."""
    import numpy as np
    from oracle import oracle_from_workload, states_to_f64
    from synth import make_prompt_states, make_prompt_tokens, make_step_states, make_step_tokens

    orc = oracle_from_workload(wl, W)
    t_total, tok, done = 0.0, 0, []
    emb = getattr(wl, "input_embed", False)
    for i in range(len(lens)):
        st = states_to_f64(make_prompt_states(wl, lens, requests=[i]), wl.act_fmt)
        sp = states_to_f64(make_step_states(wl, len(lens), 1, requests=[i]), wl.act_fmt)
        tp = make_prompt_tokens(wl, lens, requests=[i]) if emb else None
        ts = make_step_tokens(wl, len(lens), 1, requests=[i]) if emb else None
        t0 = time.perf_counter()
        _, _, s = orc.prefill([int(lens[i])], *st, tokens=tp)
        orc.step(s, *sp, tokens=ts)
        t_total += time.perf_counter() - t0
        tok += int(lens[i]) + 1
        done.append(i)
        if t_total >= budget_s:
            break
    tok_per_s = tok / t_total
    mean_tokens = (float(np.sum(lens)) + len(lens)) / len(lens)
    threads = None
    try:
        from threadpoolctl import threadpool_info
        threads = max((p.get("num_threads") or 0) for p in threadpool_info()) or None
    except Exception:
        pass
    return {
        "value": tok_per_s / mean_tokens,
        "unit": "requests/s",
        "cores": threads or os.cpu_count(),
        "blas_threads": threads,
        "host_cpus": os.cpu_count(),
        "kind": "oracle",
        "sample": f"requests {done[0]}..{done[-1]} of the batch ({len(done)} requests, {tok} tokens, "
                  f"prefill + 1 step each, fp64 numpy, {t_total:.1f} s); rate scaled by the batch's "
                  f"mean of {mean_tokens:.0f} tokens per request",
        "draft_tokens_per_s": tok_per_s,
    }


def _emit(out):
    print(json.dumps(out), flush=True)
    return 0


def decode_step_bytes(shape, n_req: int, keys: float, weight_bytes: float) -> float:
    """Algorithmic HBM bytes of one decode step: every cached key and value
    read once (plus the new token's K/V written), the weights read once, the
    three input state rows, the running pool sums read and written, z out."""
    kv_read = keys * shape.n_kv * shape.head_dim * 2 * 2
    kv_write = n_req * shape.n_kv * shape.head_dim * 2 * 2
    states = n_req * 3 * shape.d * 2
    pool = n_req * shape.d * 4 * 2
    return kv_read + kv_write + weight_bytes + states + pool + 4 * n_req


def weight_bytes(W) -> float:
    """Bytes of every stored weight tensor (codes and row scales for e4m3)."""
    import numpy as np
    total = 0
    for k, v in W.items():
        if k == "_fmt":
            continue
        for arr in (v if isinstance(v, tuple) else (v,)):
            total += np.asarray(arr).nbytes
    return float(total)


def measure_decode(seed: int, steps: int, warmup: int, attn_gate: bool = False):
    """Dynamic re-prediction at scale: 512 in-flight
    requests whose paged draft KV caches hold U[256, 8192] prompt tokens
    (filled by untimed prefill calls), then ``steps`` timed decode steps of
    one new token per request.  Returns the measurement as a dict."""
    import numpy as np
    import torch
    from paper_2609_01068_amd.predictor import OutletsPredictor
    from synth import device_states, make_lengths, make_weights, workload

    wl = workload(3, attn_gate=attn_gate)
    print(f"[bench] generating {wl.name} weights", file=sys.stderr, flush=True)
    W = make_weights(wl, seed)
    wbytes = weight_bytes(W)
    lens = make_lengths(wl, seed)
    B = len(lens)
    max_seq = int(lens.max()) + steps + warmup + 16
    pages = int(sum((int(n) + steps + warmup + 15) // 16 for n in lens)) + B
    chunk = 48
    max_chunk_tokens = max(int(lens[i:i + chunk].sum()) for i in range(0, B, chunk))
    pred = OutletsPredictor(wl.shape, wl.weight_fmt, wl.act_fmt, W, max_slots=B, max_seq_len=max_seq,
                            num_pages=pages, max_batch_tokens=max_chunk_tokens, max_batch_requests=B)
    del W
    print(f"[bench] filling {B} KV caches ({int(lens.sum())} tokens) with prefill calls", file=sys.stderr, flush=True)
    for i in range(0, B, chunk):
        idx = list(range(i, min(B, i + chunk)))
        H = device_states(wl, int(lens[idx].sum()), seed, 300, i)
        pred.prefill(idx, lens[idx], *H)
        torch.cuda.synchronize()
        del H
    print(f"[bench]   caches filled; warmup {warmup}, timed {steps} decode steps", file=sys.stderr, flush=True)
    n_in = warmup + steps
    S = [device_states(wl, B, seed, 400, t) for t in range(n_in)]
    slots = list(range(B))
    z = torch.empty(B, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    for t in range(warmup):
        pred.step(slots, *S[t], z_out=z, stream=stream)
    torch.cuda.synchronize()
    cached0 = int(lens.sum()) + B * warmup
    # timed region: events around the dominant kernel only (timing every
    # kernel group costs ~0.09 ms per step)
    pred.profile(True, groups=["ATTN"])
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for t in range(warmup, n_in):
        pred.step(slots, *S[t], z_out=z, stream=stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    prof = pred.profile_read("step")
    # per-group breakdown from two further (untimed) steps with every group timed
    pred.profile(True)
    for t in range(2):
        pred.step(slots, *S[t], z_out=z, stream=stream)
    breakdown = pred.profile_read("step")
    pred.profile(False)
    pred.close()
    ms_per_step = max(gpu_ms, wall * 1e3) / steps
    # keys read per step: every cached token of every request plus the new one
    keys = sum(cached0 + B * (t + 1) for t in range(steps)) / steps
    kv_bytes = keys * wl.shape.n_kv * wl.shape.head_dim * 2 * 2
    attn_ms = prof["ATTN"][0] / max(1, prof["ATTN"][1])
    attn_gbs = kv_bytes / (attn_ms * 1e-3) / 1e9
    step_bytes = decode_step_bytes(wl.shape, B, keys, wbytes)
    step_gbs = step_bytes / (ms_per_step * 1e-3) / 1e9
    return {
        "wl": wl, "requests": B, "steps": steps, "warmup": warmup, "ms_per_step": ms_per_step,
        "draft_tokens_per_s": B / (ms_per_step / 1e3), "cached_tokens_at_start": cached0,
        "attn": {"kernel": "decode attention over the paged KV cache", "bound": "hbm", "achieved": attn_gbs,
                 "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": attn_gbs / PEAK_HBM_GBS,
                 "traffic": recorded_traffic("decode_attention_8b_b512.md", "attn.hip", "attn"),
                 "bytes_per_launch": kv_bytes, "avg_ms": attn_ms},
        "step": {"bound": "hbm", "achieved": step_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                 "frac": step_gbs / PEAK_HBM_GBS, "bytes_per_step": step_bytes, "kv_bytes_per_step": kv_bytes,
                 "weight_bytes": wbytes},
        "kernels_step": {n: {"avg_ms": ms / k, "launches": k} for n, (ms, k) in breakdown.items() if k},
    }


def bench_decode(a):
    """The 512-request decode steps as the bench line itself."""
    m = measure_decode(a.seed, a.steps, a.warmup, a.attn_gate)
    out = {
        "metric": METRIC, "value": m["draft_tokens_per_s"], "unit": "draft tokens/s (request-steps/s)",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": m["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded on device; U[256,8192] cached prompt tokens; fresh N(0,1) x (1,4,16) states per step)",
        "config": {"workload": DECODE_WORKLOAD, "requests": m["requests"],
                   "cached_tokens_at_start": m["cached_tokens_at_start"], "attn_gate": m["wl"].attn_gate},
        "roofline": m["attn"],
        "step_hbm": m["step"],
        "kernels_step": m["kernels_step"],
        "kernels_note": "per-group times from 2 untimed steps with every group timed",
    }
    return _emit(out)


DECODE_WORKLOAD = ("8B-shaped bf16 draft layer + length head, dynamic re-prediction: 512 in-flight requests "
                   "with paged draft KV caches of U[256, 8192] tokens (page 16), one new token per request per step")


def bench_prefill(a, cfg_id):
    """Static prediction of one large batch in a single call (configs 2 and 4)."""
    import numpy as np
    import torch
    from paper_2609_01068_amd.predictor import OutletsPredictor, to_device
    from synth import device_states, make_lengths, make_weights, workload

    wl = workload(cfg_id, attn_gate=a.attn_gate)
    print(f"[bench] generating {wl.name} weights and inputs", file=sys.stderr, flush=True)
    W = make_weights(wl, a.seed)
    lens = make_lengths(wl, a.seed)
    T, B = int(lens.sum()), len(lens)
    H = device_states(wl, T, a.seed, 300, 0)
    pred = OutletsPredictor(wl.shape, wl.weight_fmt, wl.act_fmt, W, max_slots=B,
                            max_seq_len=int(lens.max()) + 16, num_pages=B * ((int(lens.max()) + 31) // 16),
                            max_batch_tokens=T, max_batch_requests=B)
    del W
    print(f"[bench] {B} requests, {T} tokens; warmup {a.warmup}, timed {a.steps}", file=sys.stderr, flush=True)
    slots = list(range(B))
    z = torch.empty(B, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    for _ in range(a.warmup):
        pred.prefill(slots, lens, *H, z_out=z, stream=stream)
        pred.release(slots)
    torch.cuda.synchronize()
    dom = "GATE_UP_GEMM"
    pred.profile(True, groups=[dom])      # timed region: the dominant kernel only
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(a.steps):
        pred.prefill(slots, lens, *H, z_out=z, stream=stream)
        pred.release(slots)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    prof = pred.profile_read("prefill")
    pred.profile(True)                    # per-group breakdown: one further untimed call
    pred.prefill(slots, lens, *H, z_out=z, stream=stream)
    pred.release(slots)
    breakdown = pred.profile_read("prefill")
    pred.profile(False)
    ms_per_step = max(ev0.elapsed_time(ev1), wall * 1e3) / a.steps
    flops = gemm_flops(wl.shape, T, wl.attn_gate, wl.input_embed)
    kernels = {}
    for name, (ms, n) in breakdown.items():
        if n:
            kernels[name] = {"avg_ms": ms / n, "launches": n}
            if name in flops:
                kernels[name]["tflops"] = flops[name] / (ms / n * 1e-3) / 1e12
    dom_ms = prof[dom][0] / max(1, prof[dom][1])
    achieved = flops[dom] / (dom_ms * 1e-3) / 1e12
    out = {
        "metric": METRIC, "value": B / (ms_per_step / 1e3), "unit": "requests/s", "n_gpus": 1,
        "steps": a.steps, "warmup": a.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16" if wl.weight_fmt == "bf16" else "bf16 (e4m3 weights)",
        "data": "synthetic (seeded; lognormal prompt lengths; N(0,1) x (1,4,16) target states drawn on device)",
        "config": {"workload": wl.name, "requests": B, "prompt_tokens": T, "d": wl.shape.d,
                   "heads": [wl.shape.n_q, wl.shape.n_kv], "ffn": wl.shape.ffn, "weights": wl.weight_fmt,
                   "attn_gate": wl.attn_gate},
        "draft_tokens_per_s": T / (ms_per_step / 1e3),
        "roofline": {"kernel": "gate/up GEMM + SwiGLU epilogue (prefill)", "bound": "mfma",
                     "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None, "avg_ms": dom_ms},
        "kernels_prefill": kernels,
        "kernels_note": "per-group times from one untimed call with every group timed",
    }
    if wl.weight_fmt == "e4m3":
        # the e4m3 weights are widened to bf16 exactly and multiplied on the
        # bf16 MFMA; the fp8 MFMA peak is reported beside the bf16 one
        out["roofline"]["peak_fp8"] = PEAK_FP8_TFLOPS
        out["roofline"]["frac_fp8_peak"] = achieved / PEAK_FP8_TFLOPS
    pred.close()
    return _emit(out)


def bench_probe(a):
    """The MLP-probe baseline on the 32-request 8B batch: probe prefill over the
    mid-depth target state of 32 requests + one probe step + release."""
    import torch
    from paper_2609_01068_amd.predictor import OutletsPredictor, to_device
    from synth import device_states, make_lengths, make_probe_weights, make_weights, workload

    wl = workload(1)
    print(f"[bench] generating {wl.name} probe weights and inputs", file=sys.stderr, flush=True)
    W = make_weights(wl, a.seed)
    PW = make_probe_weights(wl, a.seed)
    W.update({k: v for k, v in PW.items() if k != "_fmt"})
    lens = make_lengths(wl, a.seed)
    T, B = int(lens.sum()), len(lens)
    h = device_states(wl, T, a.seed, 300, 0)[1]
    hs = device_states(wl, B, a.seed, 400, 1)[1]
    pred = OutletsPredictor(wl.shape, wl.weight_fmt, wl.act_fmt, W, max_slots=B, max_seq_len=16,
                            num_pages=1, max_batch_tokens=T, max_batch_requests=B)
    del W
    slots = list(range(B))
    z = torch.empty(B, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    def step():
        pred.probe_prefill(slots, lens, h, z_out=z, stream=stream)
        pred.probe_step(slots, hs, z_out=z, stream=stream)
        pred.probe_release(slots)
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(a.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = ev0.elapsed_time(ev1) / a.steps
    ms_per_step = max(ev_ms, wall * 1e3 / a.steps)
    in_bytes = (T + B) * wl.shape.d * 2 + 2 * wl.shape.head_hidden * 2 * wl.shape.d * 2
    achieved = in_bytes / (ev_ms * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": B / (ms_per_step / 1e3), "unit": "requests/s", "n_gpus": 1,
        "steps": a.steps, "warmup": a.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded; lognormal prompt lengths; N(0,1) x 4 mid-depth target states drawn on device)",
        "config": {"workload": "MLP-probe baseline on the 32-request 8B batch: probe prefill on the "
                               "mid-depth state + one probe step per request", "requests": B, "prompt_tokens": T,
                   "d": wl.shape.d, "head_hidden": wl.shape.head_hidden},
        "roofline": {"kernel": "probe call (pooling + head), whole step", "bound": "hbm", "achieved": achieved,
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": None,
                     "bytes_per_step": in_bytes, "avg_ms": ev_ms},
    }
    pred.close()
    return _emit(out)


def bench_sched(a):
    """The control plane that consumes the static prediction (Section 5
    system evaluation) on the saturation trace: one step = whole-token
    predictions from z_hat, the LB + SJF decode-cluster simulation of all
    1,914 requests, and its serving metrics.  Host code only (no GPU)."""
    import numpy as np
    from paper_2609_01068_amd import binding as B
    from synth.serving import PAPER_TRACE as tr, make_trace, noisy_predictions

    arrival, L = make_trace(tr, a.seed)
    noisy = noisy_predictions(L, 0.25, a.seed)
    z = np.log1p(noisy.astype(np.float64)).astype(np.float32)
    cluster = (tr.instances, tr.max_running)
    it = (tr.iter_base_us, tr.iter_per_seq_us)

    def one_step():
        p = B.outlets_pred_tokens(z)
        _, _, fin = B.outlets_sched_simulate(arrival, L, p, *cluster, B.OUTLETS_ROUTE_LB,
                                             B.OUTLETS_QUEUE_SJF, *it)
        return B.outlets_sched_metrics(arrival, L, fin)

    for _ in range(a.warmup):
        one_step()
    t0 = time.perf_counter()
    for _ in range(a.steps):
        one_step()
    wall = time.perf_counter() - t0
    ms = wall * 1e3 / a.steps

    def row(routing, order, pred):
        _, _, fin = B.outlets_sched_simulate(arrival, L, pred, *cluster, routing, order, *it)
        m = B.outlets_sched_metrics(arrival, L, fin)
        return {"tokens_per_s": m[0], "mean_latency_s": m[1], "p99_short_s": m[2], "p99_medium_s": m[3],
                "p99_long_s": m[4], "makespan_s": m[5]}
    RR, LB, FCFS, SJF = B.OUTLETS_ROUTE_RR, B.OUTLETS_ROUTE_LB, B.OUTLETS_QUEUE_FCFS, B.OUTLETS_QUEUE_SJF
    p_tok = B.outlets_pred_tokens(z)
    serving = {
        "RR+FCFS": row(RR, FCFS, p_tok),
        "RR+SJF": row(RR, SJF, p_tok),
        "LB+SJF": row(LB, SJF, p_tok),
        "RR+SJF exact lengths": row(RR, SJF, L),
        "LB+SJF exact lengths": row(LB, SJF, L),
    }
    out = {
        "metric": "control plane: requests predicted-length-converted, routed (LB) and queued (SJF) through "
                  "a full decode-cluster simulation, per host second",
        "value": tr.n / (ms / 1e3), "unit": "requests/s (host)", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "int64",
        "data": "synthetic (seeded Poisson arrivals at 100/s, lognormal output lengths, median 1,030, "
                "sigma 0.6, clipped to 2,047; predictions with lognormal error sigma 0.25)",
        "config": {"workload": "1P3D decode cluster, 3 instances x 256 slots, iteration 12 ms + 0.12 ms per "
                               "running request, 1,914 requests", "requests": tr.n,
                   "mean_output_tokens": float(L.mean()),
                   "prediction_mae_tokens": float(np.abs(p_tok.astype(np.int64) - L).mean())},
        "roofline": None,
        "serving": serving,
    }
    if not a.no_cpu_baseline:
        from oracle import sched as S
        t0 = time.perf_counter()
        S.simulate([int(x) for x in arrival], [int(x) for x in L], S.pred_tokens(z), *cluster, S.LB, S.SJF, *it)
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": tr.n / dt, "unit": "requests/s (host)", "cores": 1, "kind": "oracle",
                               "sample": f"one LB+SJF simulation of the whole trace in plain Python ({dt:.2f} s)"}
    return _emit(out)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--decode-steps", type=int, default=20,
                    help="prefill-8b: timed 512-request decode steps reported under decode_step")
    ap.add_argument("--no-decode", action="store_true",
                    help="prefill-8b: skip the 512-request decode-step measurement")
    ap.add_argument("--workload", default="prefill-8b",
                    choices=["prefill-8b", "decode-8b", "prefill-8b-large", "prefill-70b-e4m3", "probe-8b",
                             "sched-1p3d"],
                    help="prefill-8b (default): 32-request 8B prefill + one step; decode-8b: 512 "
                         "in-flight requests with 256..8192 cached tokens, timed decode steps; "
                         "prefill-8b-large: 256 requests (~466k tokens) in one call; "
                         "prefill-70b-e4m3: 70B shape with e4m3 weights, 64 requests; probe-8b: the "
                         "MLP-probe baseline on the 32-request 8B batch; sched-1p3d: the LB + SJF control "
                         "plane on the 1,914-request saturation trace (host only)")
    ap.add_argument("--attn-gate", action="store_true",
                    help="draft layer with the Gated Attention output gate (Section 4.1)")
    ap.add_argument("--draft-head", action="store_true",
                    help="prefill-8b: also run the draft model head (Eq. 2, V = 128,256) after the "
                         "prefill and after the step")
    ap.add_argument("--input-embed", action="store_true",
                    help="prefill-8b: draft layer with EAGLE-3 input embeddings (QKV over [emb ; f_ctx], "
                         "V = 128,256 embedding table)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (3 times); used to scale "
                         "rocprof's FETCH_SIZE / WRITE_SIZE counters to bytes")
    a = ap.parse_args(argv)
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {a.gpus}); the path shards over "
              "requests, and this benchmark measures one GPU's share", file=sys.stderr)
        return 2

    if a.input_embed and a.workload != "prefill-8b":
        print("--input-embed is measured on the prefill-8b workload only", file=sys.stderr)
        return 2

    if a.workload == "sched-1p3d":
        return bench_sched(a)

    import numpy as np
    import torch

    if a.copy_probe:
        n = 1 << 30
        x = torch.ones(n, dtype=torch.uint8, device="cuda")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_per_launch": n, "launches": 3}))
        return 0

    from paper_2609_01068_amd.predictor import OutletsPredictor, to_device
    from synth import make_lengths, make_prompt_states, make_step_states, make_weights, workload

    if a.workload == "decode-8b":
        return bench_decode(a)
    if a.workload == "probe-8b":
        return bench_probe(a)
    if a.workload != "prefill-8b":
        return bench_prefill(a, {"prefill-8b-large": 2, "prefill-70b-e4m3": 4}[a.workload])

    wl = workload(1, attn_gate=a.attn_gate, input_embed=a.input_embed)
    print(f"[bench] generating {wl.name} weights and inputs", file=sys.stderr, flush=True)
    W = make_weights(wl, a.seed)
    if a.draft_head:
        from synth import make_lm_weights
        W["w_lm"] = make_lm_weights(wl, a.seed)["w_lm"]
    lens = make_lengths(wl, a.seed)
    T, B = int(lens.sum()), len(lens)
    H = [to_device(x) for x in make_prompt_states(wl, lens, a.seed)]
    S = [to_device(x) for x in make_step_states(wl, B, 1, a.seed)]
    tok_p = tok_step = None
    if wl.input_embed:
        from synth import make_prompt_tokens, make_step_tokens
        tok_p = torch.from_numpy(make_prompt_tokens(wl, lens, a.seed)).cuda()
        tok_step = torch.from_numpy(make_step_tokens(wl, B, 1, a.seed)).cuda()
    pred = OutletsPredictor(wl.shape, wl.weight_fmt, wl.act_fmt, W, max_slots=B,
                            max_seq_len=int(lens.max()) + 16, num_pages=B * ((int(lens.max()) + 16 + 15) // 16),
                            max_batch_tokens=T, max_batch_requests=B)
    slots = list(range(B))
    z = torch.empty(B, dtype=torch.float32, device="cuda")
    z1 = torch.empty(B, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    probs = torch.empty((B, wl.shape.vocab), dtype=torch.float32, device="cuda") if a.draft_head else None

    def one_step():
        pred.prefill(slots, lens, *H, z_out=z, stream=stream, tokens=tok_p)
        if probs is not None:
            pred.draft_distribution(B, p_out=probs, stream=stream)
        pred.step(slots, *S, z_out=z1, stream=stream, tokens=tok_step)
        if probs is not None:
            pred.draft_distribution(B, p_out=probs, stream=stream)
        pred.release(slots)

    print(f"[bench] warmup {a.warmup} steps (T={T} tokens, B={B})", file=sys.stderr, flush=True)
    for _ in range(a.warmup):
        one_step()
    torch.cuda.synchronize()
    dom = "GATE_UP_GEMM"
    pred.profile(True, groups=[dom])      # timed region: events around the dominant kernel only
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(a.steps):
        one_step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    prof_dom = pred.profile_read("prefill")[dom]
    pred.profile(True)                    # per-group breakdown: two further untimed steps
    for _ in range(2):
        one_step()
    prof_pre = pred.profile_read("prefill")
    prof_step = pred.profile_read("step")
    pred.profile(False)
    print(f"[bench] timed {a.steps} steps: {gpu_ms:.2f} ms (events), {wall * 1e3:.2f} ms (wall)",
          file=sys.stderr, flush=True)
    ms_per_step = max(gpu_ms, wall * 1e3) / a.steps
    req_s = B / (ms_per_step / 1e3)
    tok_s = (T + B) / (ms_per_step / 1e3)

    flops = gemm_flops(wl.shape, T, wl.attn_gate, wl.input_embed)
    kernels = {}
    for name, (ms, n) in prof_pre.items():
        if n:
            kernels[name] = {"avg_ms": ms / n, "launches": n}
            if name in flops:
                kernels[name]["tflops"] = flops[name] / (ms / n * 1e-3) / 1e12
    dom_ms = prof_dom[0] / max(1, prof_dom[1])
    achieved = flops[dom] / (dom_ms * 1e-3) / 1e12
    step_kernels = {name: {"avg_ms": ms / n, "launches": n} for name, (ms, n) in prof_step.items() if n}

    out = {
        "metric": METRIC,
        "value": req_s,
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; lognormal prompt lengths; N(0,1) x (1,4,16) target states; N(0,0.02) weights)",
        "config": {"workload": "8B-shaped bf16 draft layer + length head: 32 requests, lognormal(512, 1.0) "
                               "prompts clipped to [32, 4096], static prediction + 1 dynamic step per request",
                   "requests": B, "prompt_tokens": T, "d": wl.shape.d, "heads": [wl.shape.n_q, wl.shape.n_kv],
                   "head_dim": wl.shape.head_dim, "ffn": wl.shape.ffn, "head_hidden": wl.shape.head_hidden,
                   "page_size": 16, "attn_gate": wl.attn_gate, "input_embed": wl.input_embed,
                   "draft_head_vocab": wl.shape.vocab if a.draft_head else 0},
        "draft_tokens_per_s": tok_s,
        "roofline": {"kernel": "gate/up GEMM + SwiGLU epilogue (prefill)", "bound": "mfma",
                     "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": recorded_traffic(),
                     "flops_per_launch": flops[dom], "avg_ms": dom_ms},
        "kernels_prefill": kernels,
        "kernels_step": step_kernels,
        "kernels_note": "per-group times from 2 untimed steps with every group timed",
    }
    pred.close()
    del H, S
    if not a.no_decode:
        # the decode-step half of the metric (512 in-flight
        # requests, HBM-bound): ms per step, draft tokens/s, the attention
        # kernel's and the whole step's fraction of the HBM peak
        m = measure_decode(a.seed, a.decode_steps, a.warmup, a.attn_gate)
        out["decode_step"] = {
            "workload": DECODE_WORKLOAD, "requests": m["requests"], "steps": m["steps"],
            "warmup": m["warmup"], "cached_tokens_at_start": m["cached_tokens_at_start"],
            "ms_per_step": m["ms_per_step"], "draft_tokens_per_s": m["draft_tokens_per_s"],
            "attention_hbm": m["attn"], "step_hbm": m["step"], "kernels_step": m["kernels_step"],
        }
    if not a.no_cpu_baseline:
        print("[bench] timing the fp64 oracle on a sample (cpu_baseline)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, W, lens, a.cpu_budget)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
