"""Parity at the benchmark configurations' full sizes (MI355X).

The GPU runs the whole batch in the launch configuration bench.py times; the
fp64 oracle recomputes a sample of requests one by one.  Sampled requests use
host-drawn states the oracle reproduces; the rest of the batch uses
on-device draws.  Tolerances as in test_gpu_parity.py.
"""
import numpy as np
import pytest

from gpu_common import (TOL_HDRAFT, TOL_Z, mixed_prompt_states, mixed_step_states, oracle_for,
                        oracle_states, rel_fro, require_gpu, say, tensor_to_f64)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _check_prefill_sample(wl, W, lens, z, hd, sample, fmt):
    from oracle import oracle_from_workload, states_to_f64
    from synth import make_prompt_states
    orc = oracle_from_workload(wl, W)
    off = np.concatenate([[0], np.cumsum(lens)])
    zg = tensor_to_f64(z)
    floor = float(np.sqrt(np.mean(zg ** 2)))
    states = {}
    for i in sample:
        O = states_to_f64(make_prompt_states(wl, lens, requests=[i]), wl.act_fmt)
        zi, hi, st = orc.prefill_one(*O)
        states[i] = st
        err = rel_fro(tensor_to_f64(hd[off[i]:off[i + 1]]), hi)
        dz = abs(zg[i] - zi) / max(abs(zi), floor)
        say(f"  request {i} (n={int(lens[i])}): h_draft rel err {err:.3e}, z rel err {dz:.3e}")
        assert err <= TOL_HDRAFT[fmt]
        assert dz <= TOL_Z[fmt]
    return orc, states


def _predictor(wl, W, lens, max_batch_tokens=None, extra=16):
    from paper_2609_01068_amd.predictor import OutletsPredictor
    B = len(lens)
    max_seq = int(lens.max()) + extra
    return OutletsPredictor(wl.shape, wl.weight_fmt, wl.act_fmt, W, max_slots=B, max_seq_len=max_seq,
                            num_pages=int(sum((int(n) + extra + 15) // 16 for n in lens)) + B,
                            max_batch_tokens=max_batch_tokens or int(lens.sum()), max_batch_requests=B)


def test_config2_saturated_prefill_256_requests():
    from synth import make_lengths, make_weights, workload
    wl = workload(2)
    lens = make_lengths(wl)
    order = np.argsort(lens)
    sample = [int(order[0]), int(order[len(order) // 4])]
    say(f"case: config-2 8B bf16, B={len(lens)}, T={int(lens.sum())} in one call, oracle on requests {sample}")
    W = make_weights(wl)
    H = mixed_prompt_states(wl, lens, sample)
    say("  inputs generated")
    pred = _predictor(wl, W, lens)
    z, hd = pred.prefill(list(range(len(lens))), lens, *H, want_hdraft=True)
    assert np.all(np.isfinite(tensor_to_f64(z)))
    say("  GPU prefill done; running the oracle")
    _check_prefill_sample(wl, W, lens, z, hd, sample, "bf16")
    pred.close()


def test_config4_70b_e4m3_prefill_64_requests():
    from synth import make_lengths, make_weights, workload
    wl = workload(4)
    lens = make_lengths(wl)
    order = np.argsort(lens)
    sample = [int(order[0])]
    say(f"case: config-4 70B e4m3 weights, B={len(lens)}, T={int(lens.sum())} in one call, oracle on request {sample}")
    W = make_weights(wl)
    say("  weights generated")
    H = mixed_prompt_states(wl, lens, sample)
    pred = _predictor(wl, W, lens)
    z, hd = pred.prefill(list(range(len(lens))), lens, *H, want_hdraft=True)
    assert np.all(np.isfinite(tensor_to_f64(z)))
    say("  GPU prefill done; running the oracle")
    _check_prefill_sample(wl, W, lens, z, hd, sample, "e4m3")
    pred.close()


def test_config3_decode_512_slots_long_caches():
    import torch
    from synth import make_lengths, make_weights, workload
    wl = workload(3)
    lens = make_lengths(wl)
    B = len(lens)
    order = np.argsort(lens)
    sample = [int(order[0]), int(order[B // 8])]   # one short cache, one of several decode chunks
    steps = 3
    say(f"case: config-3 8B bf16, {B} slots, {int(lens.sum())} cached tokens, {steps} steps, oracle on slots {sample}")
    W = make_weights(wl)
    chunk = 48
    max_chunk = max(int(lens[i:i + chunk].sum()) for i in range(0, B, chunk))
    pred = _predictor(wl, W, lens, max_batch_tokens=max_chunk, extra=steps + 16)
    z_pre, hd_pre = {}, {}
    for i in range(0, B, chunk):
        idx = list(range(i, min(B, i + chunk)))
        sub = [j for j in idx if j in sample]
        H = mixed_prompt_states(wl, lens[idx], [])
        # sampled requests use their own host draws (generator index = batch index)
        if sub:
            from paper_2609_01068_amd.predictor import to_device
            from synth import make_prompt_states
            off = np.concatenate([[0], np.cumsum(lens[idx])])
            for j in sub:
                k = idx.index(j)
                S = make_prompt_states(wl, lens, requests=[j])
                for d in range(3):
                    H[d][off[k]:off[k + 1]] = to_device(S[d])
        z, hd = pred.prefill(idx, lens[idx], *H, want_hdraft=True)
        off = np.concatenate([[0], np.cumsum(lens[idx])])
        for j in sub:
            k = idx.index(j)
            z_pre[j] = float(z[k])
            hd_pre[j] = tensor_to_f64(hd[off[k]:off[k + 1]])
        torch.cuda.synchronize()
        say(f"  prefilled slots {idx[0]}..{idx[-1]}")
    from oracle import oracle_from_workload, states_to_f64
    from synth import make_prompt_states, make_step_states
    orc = oracle_from_workload(wl, W)
    states = {}
    for j in sample:
        zi, hi, st = orc.prefill_one(*states_to_f64(make_prompt_states(wl, lens, requests=[j]), wl.act_fmt))
        states[j] = st
        assert rel_fro(hd_pre[j], hi) <= TOL_HDRAFT["bf16"]
    slots = list(range(B))
    for t in range(1, steps + 1):
        S = mixed_step_states(wl, B, t, sample)
        z, hd = pred.step(slots, *S, want_hdraft=True)
        zg, hg = tensor_to_f64(z), tensor_to_f64(hd)
        floor = float(np.sqrt(np.mean(zg ** 2)))
        for j in sample:
            sj = states_to_f64(make_step_states(wl, B, t, requests=[j]), wl.act_fmt)
            zr, hr = orc.step_one(states[j], sj[0][0], sj[1][0], sj[2][0])
            err, dz = rel_fro(hg[j], hr), abs(zg[j] - zr) / max(abs(zr), floor)
            say(f"  step {t} slot {j}: h_draft rel err {err:.3e}, z rel err {dz:.3e}")
            assert err <= TOL_HDRAFT["bf16"]
            assert dz <= TOL_Z["bf16"]
    pred.close()
