"""outlets_predict_step_noalloc (per-call buffers in the library's static
scratch array) against outlets_predict_step (MI355X, through the C ABI).

Two contexts with the same weights and history: one steps through
outlets_predict_step, the other through the no-allocation entry point.  The
two take the same kernels and split plans, so z and h_draft must agree bit
for bit, on two calls in a row, the second with fewer requests (the scratch
keeps the first call's contents).  Also: the refusals (oversized call with
the state unchanged, kept intermediates) and that per-call inspection is
refused after a no-allocation step.
"""
import numpy as np
import pytest

from gpu_common import device_states, make_case, make_predictor, reduced_shape, require_gpu, say, step_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _pair(case, max_seq_len):
    n = len(case.lens)
    pa = make_predictor(case, max_slots=n, max_seq_len=max_seq_len)
    pb = make_predictor(case, max_slots=n, max_seq_len=max_seq_len)
    H = device_states(case)
    pa.prefill(list(range(n)), case.lens, *H)
    pb.prefill(list(range(n)), case.lens, *H)
    return pa, pb


def _compare_steps(case, pa, pb, batches):
    import torch
    for t, slots in enumerate(batches, start=1):
        S = [x[slots].contiguous() for x in device_states(case, step_inputs(case, t))]
        za, ha = pa.step(slots, *S, want_hdraft=True)
        z = torch.empty(len(slots), dtype=torch.float32, device="cuda")
        h = torch.empty((len(slots), case.wl.shape.d), dtype=pa.act_dtype, device="cuda")
        zb, hb = pb.step(slots, *S, z_out=z, hdraft_out=h, noalloc=True)
        torch.cuda.synchronize()
        same_z = torch.equal(za, zb)
        same_h = torch.equal(ha, hb)
        say(f"  call {t}: {len(slots)} requests, z bit-identical {same_z}, h_draft bit-identical {same_h}")
        assert same_z and same_h, t
    from paper_2609_01068_amd import binding as B
    assert np.array_equal(pa.meta(B.OUTLETS_META_SEQ_LEN), pb.meta(B.OUTLETS_META_SEQ_LEN))
    assert np.array_equal(pa.meta(B.OUTLETS_META_PAGE_TABLE), pb.meta(B.OUTLETS_META_PAGE_TABLE))


def test_noalloc_step_matches_step_8b_shape():
    """8B shape: 96 caches of 40..1,500 tokens, then a call of 96 requests
    (128-row tiles, K splits in the shared partial region, multi-chunk
    split-KV attention) and one of 33 (64-row tiles)."""
    n = 96
    lens = [40 + (97 * i) % 1461 for i in range(n)]
    case = make_case(1, lens=lens, n_req=n)
    say(f"case: 8B bf16, {n} caches of {min(lens)}..{max(lens)} tokens; step vs no-allocation step, "
        f"calls of {n} then 33 requests")
    pa, pb = _pair(case, max(lens) + 8)
    _compare_steps(case, pa, pb, [list(range(n)), list(range(5, 71, 2))])
    pa.close()
    pb.close()


def test_noalloc_step_matches_step_reduced_gated():
    """bf16 d=512 8q/2kv with the Gated Attention gate: 7 requests then 3."""
    case = make_case(1, lens=[1, 17, 300, 1100, 33, 64, 5], shape=reduced_shape(), n_req=7, attn_gate=True)
    say("case: bf16 reduced shape + gate, 7 caches; step vs no-allocation step, calls of 7 then 3 requests")
    pa, pb = _pair(case, 1200)
    _compare_steps(case, pa, pb, [list(range(7)), [6, 3, 0]])
    pa.close()
    pb.close()


def test_noalloc_step_matches_step_tiny_fp32():
    case = make_case(0)
    say("case: tiny fp32 shape, 4 requests; step vs no-allocation step, calls of 4 then 2 requests")
    pa, pb = _pair(case, 128)
    _compare_steps(case, pa, pb, [[0, 1, 2, 3], [2, 0]])
    pa.close()
    pb.close()


def test_noalloc_step_refusals_leave_state_unchanged():
    from paper_2609_01068_amd import binding as B
    n = 2048
    case = make_case(1, lens=[1] * n, n_req=n)
    say(f"case: 8B bf16, {n} one-token requests: a no-allocation step of all of them exceeds the scratch")
    pred = make_predictor(case, max_slots=n, max_seq_len=8)
    H = device_states(case)
    slots = list(range(n))
    pred.prefill(slots, case.lens, *H)
    table = pred.meta(B.OUTLETS_META_PAGE_TABLE)
    S = device_states(case, step_inputs(case, 1))
    with pytest.raises(B.OutletsError) as e:
        pred.step(slots, *S, noalloc=True)
    assert e.value.rc == B.OUTLETS_ERR_INVALID_ARG and "scratch" in str(e.value)
    assert np.array_equal(pred.meta(B.OUTLETS_META_SEQ_LEN)[:n], np.ones(n, np.int32))
    assert np.array_equal(pred.meta(B.OUTLETS_META_PAGE_TABLE), table)
    # a smaller call fits; per-call inspection is refused after it
    pred.step(slots[:256], *[x[:256] for x in S], noalloc=True)
    with pytest.raises(B.OutletsError) as e:
        pred.buffer("ATTN", pred.act_dtype)
    assert e.value.rc == B.OUTLETS_ERR_INVALID_ARG
    with pytest.raises(B.OutletsError) as e:
        pred.meta(B.OUTLETS_META_DEV_POSITIONS)
    assert e.value.rc == B.OUTLETS_ERR_INVALID_ARG
    pred.step(slots[:256], *[x[:256] for x in S])          # the ordinary step clears the refusal
    assert pred.buffer("ATTN", pred.act_dtype).numel() == 256 * case.wl.shape.n_q * case.wl.shape.head_dim
    pred.close()
    kept = make_predictor(make_case(0), keep=True)
    kept.prefill([0], [4], *[x[:4] for x in device_states(make_case(0))])
    with pytest.raises(B.OutletsError) as e:
        kept.step([0], *[x[:1] for x in device_states(make_case(0), step_inputs(make_case(0), 1))], noalloc=True)
    assert e.value.rc == B.OUTLETS_ERR_UNSUPPORTED
    kept.close()
