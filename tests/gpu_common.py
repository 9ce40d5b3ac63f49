"""Helpers shared by the GPU parity tests: build the HIP predictor and the
fp64 oracle from the same seeded synthetic inputs, and compare them."""
from __future__ import annotations

import dataclasses
import sys
from typing import Optional

import numpy as np
import pytest

from synth import (DraftShape, make_lengths, make_prompt_states, make_prompt_tokens,
                   make_step_states, make_step_tokens, make_weights, workload)
from oracle import oracle_from_workload, states_to_f64

# Tolerances: draft states as a relative Frobenius error per request, the
# predicted log-length as |dz| <= tol * max(|z_ref|, rms(z_ref)).  The
# attention output (heads concatenated, before W_o) is held to the draft-state
# bound, per request and per decode step.
TOL_HDRAFT = {"f32": 1e-4, "bf16": 2e-2, "e4m3": 6e-2}
TOL_Z = {"f32": 1e-4, "bf16": 1e-2, "e4m3": 1e-2}
TOL_ATTN = TOL_HDRAFT
# GPU-vs-GPU comparisons of the same computation through different tile or
# split plans (measured spread <= 1.1e-3 on h_draft, 6e-4 on z at the 8B shape)
TOL_VARIANT = 5e-3


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2609_01068_amd import binding
    binding.lib()          # raises if the library is missing: no fallback


def rel_fro(got: np.ndarray, ref: np.ndarray) -> float:
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def z_errors(z_got, z_ref):
    """|dz| / max(|z_ref|, rms(z_ref)), the floor taken from the oracle's values
    (for a sample of a batch: the rms over the sampled requests)."""
    z_got, z_ref = np.asarray(z_got, np.float64), np.asarray(z_ref, np.float64)
    floor = max(float(np.sqrt(np.mean(z_ref ** 2))), 1e-30)
    return np.abs(z_got - z_ref) / np.maximum(np.abs(z_ref), floor)


def tensor_to_f64(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float64).cpu().numpy()


def attention_rows(pred, rows):
    """The last call's attention output (the ATTN buffer, [T, n_q*hd]) as
    float64, only the (start, stop) row ranges in ``rows``."""
    sh = pred.shape
    buf = pred.buffer("ATTN", pred.act_dtype).view(-1, sh.n_q * sh.head_dim)
    return [tensor_to_f64(buf[a:b]) for a, b in rows]


def attention_error(got: np.ndarray, ref: np.ndarray) -> float:
    """Relative Frobenius error of one request's attention output rows."""
    return rel_fro(np.asarray(got).reshape(ref.shape[0], -1), np.asarray(ref).reshape(ref.shape[0], -1))


def check_attention(got_rows, refs, fmt, label=""):
    """Every request's attention output within TOL_ATTN; returns the worst error."""
    worst = 0.0
    for i, (g, r) in enumerate(zip(got_rows, refs)):
        e = attention_error(g, r)
        worst = max(worst, e)
        assert e <= TOL_ATTN[fmt], (label, i, e)
    return worst



@dataclasses.dataclass
class Case:
    wl: object
    weights: dict
    lens: np.ndarray
    states: list            # stored (low, mid, high) packed
    fmt: str
    tokens: Optional[np.ndarray] = None    # packed int32 token ids (input embeddings)


def make_case(cfg_id: int, lens=None, seed: int = 0, **overrides) -> Case:
    wl = workload(cfg_id, **overrides)
    W = make_weights(wl, seed)
    if lens is None:
        lens = make_lengths(wl, seed)
    lens = np.asarray(lens, dtype=np.int32)
    st = make_prompt_states(wl, lens, seed)
    tok = make_prompt_tokens(wl, lens, seed) if wl.input_embed else None
    return Case(wl, W, lens, st, wl.weight_fmt, tok)


def make_predictor(case: Case, *, max_slots=None, num_pages=None, max_seq_len=None,
                   max_batch_tokens=None, max_batch_requests=None, keep=False):
    from paper_2609_01068_amd.predictor import OutletsPredictor
    wl, lens = case.wl, case.lens
    T = int(lens.sum())
    n = len(lens)
    max_seq = max_seq_len or int(lens.max()) + 64
    slots_n = max_slots or max(n, 1)
    pages = num_pages or (slots_n * (-(-max_seq // 16)))
    return OutletsPredictor(wl.shape, wl.weight_fmt, wl.act_fmt, case.weights,
                            max_slots=slots_n, max_seq_len=max_seq, num_pages=pages,
                            max_batch_tokens=max_batch_tokens or max(T, 1),
                            max_batch_requests=max_batch_requests or max(n, 1),
                            keep_intermediates=keep)


def device_states(case: Case, arrays=None):
    from paper_2609_01068_amd.predictor import to_device
    arrays = case.states if arrays is None else arrays
    return [to_device(a) for a in arrays]


def oracle_for(case: Case):
    return oracle_from_workload(case.wl, case.weights)


def oracle_states(case: Case, arrays=None):
    return states_to_f64(case.states if arrays is None else arrays, case.wl.act_fmt)


def step_inputs(case: Case, step: int, requests=None):
    return make_step_states(case.wl, len(case.lens), step, requests=requests)


def step_tokens(case: Case, step: int, requests=None):
    """Token ids of decode step ``step`` (None without input embeddings)."""
    if not case.wl.input_embed:
        return None
    return make_step_tokens(case.wl, len(case.lens), step, requests=requests)


def device_tokens(arr):
    import torch
    if arr is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.int32)).cuda()


def reduced_shape(d=512, n_q=8, n_kv=2, hd=128, ffn=1024, head_hidden=256, theta=5e5, vocab=1024):
    return DraftShape(d=d, n_q=n_q, n_kv=n_kv, head_dim=hd, ffn=ffn, head_hidden=head_hidden,
                      rope_theta=theta, vocab=vocab)


def mixed_prompt_states(wl, lens, sample, seed=0):
    """Packed prompt states for a full-size batch: requests in `sample` get the
    host draws the oracle can reproduce, the others on-device draws (their
    results are not checked; they load the call at its full size)."""
    import torch
    from paper_2609_01068_amd.predictor import to_device
    from synth import device_states, make_prompt_states
    parts = [[], [], []]
    for i, n in enumerate(lens):
        if i in sample:
            H = [to_device(x) for x in make_prompt_states(wl, lens, seed, requests=[i])]
        else:
            H = device_states(wl, int(n), seed, 300, i)
        for j in range(3):
            parts[j].append(H[j])
    return [torch.cat(p) for p in parts]


def mixed_step_states(wl, n_req, step, sample, seed=0):
    import torch
    from paper_2609_01068_amd.predictor import to_device
    from synth import device_states, make_step_states
    H = device_states(wl, n_req, seed, 400, step)
    for i in sample:
        S = make_step_states(wl, n_req, step, seed, requests=[i])
        for j in range(3):
            H[j][i:i + 1] = to_device(S[j])
    return H
