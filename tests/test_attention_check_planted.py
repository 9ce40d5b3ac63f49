"""Planted attention faults against the attention-level parity check (CPU).

The GPU parity tests compare the library's attention output (heads
concatenated, before W_o) with the oracle's for every request of every
prefill and decode step (gpu_common.check_attention).  Here plausible
kernel faults are planted in the oracle's attention and the same check is
run against the correct oracle: each fault must fail it.  The cases are
those of the GPU tests: the reduced bf16 shape with caches of 1,100 / 600 /
40 tokens (decode ranges of ~16 pages = 256 keys), and the 8B shape with
caches of 600 / 40 tokens.  On these cases the h_draft and z checks alone
let several of these faults through (the residual stream dominates
h_draft), which is why the attention output is compared directly.
"""
import dataclasses

import numpy as np
import pytest

import oracle.model as oracle_model
from gpu_common import check_attention, make_case, oracle_for, oracle_states, reduced_shape, step_inputs

REAL = oracle_model.causal_gqa_attention
CHUNK = 256          # keys per decode range at these batch sizes (~16 pages)


def _drop_first_chunk(q, k, v, q_pos, k_pos, chunk=1024):
    keep = k_pos >= CHUNK
    if keep.all() or not keep.any():
        return REAL(q, k, v, q_pos, k_pos, chunk)
    return REAL(q, k[keep], v[keep], q_pos, k_pos[keep], chunk)


def _last_chunk_only(q, k, v, q_pos, k_pos, chunk=1024):
    keep = k_pos >= (int(q_pos.max()) // CHUNK) * CHUNK
    return REAL(q, k[keep], v[keep], q_pos, k_pos[keep], chunk)


def _uniform_weights(q, k, v, q_pos, k_pos, chunk=1024):
    return REAL(np.zeros_like(q), k, v, q_pos, k_pos, chunk)


def _double_scale(q, k, v, q_pos, k_pos, chunk=1024):
    return REAL(2.0 * q, k, v, q_pos, k_pos, chunk)


def _no_mask(q, k, v, q_pos, k_pos, chunk=1024):
    return REAL(q, k, v, np.full_like(q_pos, 10 ** 9), k_pos, chunk)


def _drop_first_tile(q, k, v, q_pos, k_pos, chunk=1024):
    """Prefill: queries past the first 64-key tile never see it."""
    out = REAL(q, k, v, q_pos, k_pos, chunk)
    late = q_pos >= 64
    if late.any():
        keep = k_pos >= 64
        out[late] = REAL(q[late], k[keep], v[keep], q_pos[late], k_pos[keep], chunk)
    return out


DECODE_FAULTS = {"drop_first_chunk": _drop_first_chunk, "last_chunk_only": _last_chunk_only,
                 "uniform_weights": _uniform_weights, "double_scale": _double_scale}
PREFILL_FAULTS = {"uniform_weights": _uniform_weights, "double_scale": _double_scale,
                  "no_mask": _no_mask, "drop_first_tile": _drop_first_tile}


def _prefill(case):
    orc = oracle_for(case)
    O = oracle_states(case)
    off = np.concatenate([[0], np.cumsum(case.lens)])
    states, caps = [], []
    for i in range(len(case.lens)):
        cap = {"_only": {"attn"}}
        _, _, st = orc.prefill_one(*(x[off[i]:off[i + 1]] for x in O), capture=cap)
        states.append(st)
        caps.append(cap["attn"])
    return orc, states, caps


def _step_attention(orc, states, case):
    S = oracle_states(case, step_inputs(case, 1))
    caps = [{"_only": {"attn"}} for _ in states]
    orc.step([dataclasses.replace(st) for st in states], *S, captures=caps)
    return [c["attn"] for c in caps]


@pytest.fixture(scope="module")
def reduced():
    case = make_case(1, lens=[1100, 600, 40], shape=reduced_shape(), n_req=3)
    orc, states, pre = _prefill(case)
    return case, orc, states, pre, _step_attention(orc, states, case)


def test_correct_attention_passes_its_own_check(reduced):
    case, orc, states, pre, step = reduced
    assert check_attention(step, _step_attention(orc, states, case), "bf16") == 0.0


@pytest.mark.parametrize("fault", sorted(DECODE_FAULTS))
def test_planted_decode_faults_fail_the_attention_check(reduced, monkeypatch, fault):
    case, orc, states, _, ref = reduced
    monkeypatch.setattr(oracle_model, "causal_gqa_attention", DECODE_FAULTS[fault])
    got = _step_attention(orc, states, case)
    with pytest.raises(AssertionError):
        check_attention(got, ref, "bf16", fault)


@pytest.mark.parametrize("fault", sorted(PREFILL_FAULTS))
def test_planted_prefill_faults_fail_the_attention_check(reduced, monkeypatch, fault):
    case, _, _, ref, _ = reduced
    monkeypatch.setattr(oracle_model, "causal_gqa_attention", PREFILL_FAULTS[fault])
    _, _, got = _prefill(case)
    with pytest.raises(AssertionError):
        check_attention(got, ref, "bf16", fault)


def test_planted_dropped_chunk_fails_at_the_8b_shape(monkeypatch):
    case = make_case(1, lens=[600, 40], n_req=2)
    orc, states, _ = _prefill(case)
    ref = _step_attention(orc, states, case)
    monkeypatch.setattr(oracle_model, "causal_gqa_attention", _drop_first_chunk)
    got = _step_attention(orc, states, case)
    with pytest.raises(AssertionError):
        check_attention(got, ref, "bf16", "drop_first_chunk")
