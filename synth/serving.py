"""Seeded synthetic request traces for the decode-cluster control plane (a
stand-in for the paper's saturation test on filtered ShareGPT requests: 1,914
requests with short prompts, about 1,127 output tokens on average, under
2,048, arriving at 100 requests/s).  Input generation only."""
from __future__ import annotations

import dataclasses
from typing import Tuple

import numpy as np


@dataclasses.dataclass(frozen=True)
class ServingTrace:
    n: int = 1914                 # requests (the paper's filtered test subset)
    qps: float = 100.0            # Poisson arrival rate (saturation point of the test)
    len_median: float = 1030.0    # lognormal output lengths: mean ~1,130 after clipping
    len_sigma: float = 0.6
    len_max: int = 2047           # lengths >= 2,048 were filtered out
    instances: int = 3            # decode instances of the 1P3D cluster
    max_running: int = 256        # continuous-batching slots per instance
    iter_base_us: int = 12_000    # decode iteration: 12 ms + 0.12 ms per running request
    iter_per_seq_us: int = 120    # (~6 k tokens/s per full instance, ~18 k for three)


PAPER_TRACE = ServingTrace()


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, 7001, stream]))


def make_trace(tr: ServingTrace = PAPER_TRACE, seed: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """(arrival_us int64 [n], nondecreasing from 0; out_len int32 [n] in [1, len_max])."""
    r = _rng(seed, 0)
    gaps = np.rint(r.exponential(1e6 / tr.qps, tr.n)).astype(np.int64)
    arrival = np.cumsum(gaps) - gaps[0]
    z = r.standard_normal(tr.n)
    out_len = np.clip(np.rint(np.exp(np.log(tr.len_median) + tr.len_sigma * z)), 1, tr.len_max).astype(np.int32)
    return arrival, out_len


def noisy_predictions(out_len: np.ndarray, sigma: float, seed: int = 0) -> np.ndarray:
    """Whole-token predictions with multiplicative lognormal error:
    rint(L * exp(sigma * N(0, 1))) (sigma 0 gives the exact lengths)."""
    r = _rng(seed, 1)
    z = r.standard_normal(len(out_len))
    return np.rint(np.asarray(out_len, dtype=np.float64) * np.exp(sigma * z)).astype(np.int32)
