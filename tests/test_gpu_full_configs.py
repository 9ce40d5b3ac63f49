"""Parity at the benchmark configurations' full sizes (MI355X).

The GPU runs the whole batch in the launch configuration bench.py times; the
fp64 oracle recomputes a sample of requests one by one that always holds
each configuration's shortest and longest request.  Sampled requests use
host-drawn states the oracle reproduces; the rest of the batch uses
on-device draws.  Checked per sampled request: h_draft, z (floored on the
rms of the oracle's z over the sample) and the attention output itself, for
the prefill and for every decode step.  Tolerances as in test_gpu_parity.py.
"""
import numpy as np
import pytest

from gpu_common import (TOL_HDRAFT, TOL_Z, attention_rows, check_attention, mixed_prompt_states,
                        mixed_step_states, rel_fro, require_gpu, say, tensor_to_f64, z_errors)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _predictor(wl, W, lens, max_batch_tokens=None, extra=16):
    from paper_2609_01068_amd.predictor import OutletsPredictor
    B = len(lens)
    max_seq = int(lens.max()) + extra
    return OutletsPredictor(wl.shape, wl.weight_fmt, wl.act_fmt, W, max_slots=B, max_seq_len=max_seq,
                            num_pages=int(sum((int(n) + extra + 15) // 16 for n in lens)) + B,
                            max_batch_tokens=max_batch_tokens or int(lens.sum()), max_batch_requests=B)


def _gpu_prefill_sample(wl, W, lens, sample):
    """The whole batch in one prefill call; returns the sampled requests'
    z, h_draft rows and attention rows (host float64)."""
    H = mixed_prompt_states(wl, lens, sample)
    say("  inputs generated")
    pred = _predictor(wl, W, lens)
    z, hd = pred.prefill(list(range(len(lens))), lens, *H, want_hdraft=True)
    zg = tensor_to_f64(z)
    assert np.all(np.isfinite(zg))
    off = np.concatenate([[0], np.cumsum(lens)])
    rows = [(int(off[i]), int(off[i + 1])) for i in sample]
    out = {"z": zg[sample], "hdraft": [tensor_to_f64(hd[a:b]) for a, b in rows],
           "attn": attention_rows(pred, rows)}
    pred.close()
    del H, z, hd
    say("  GPU prefill done")
    return out


def _oracle_check(orc, wl, lens, sample, got, fmt, which):
    """Oracle prefill of the sampled requests at positions `which` of
    `sample`; compares h_draft, attention and z (z after all of them)."""
    from oracle import states_to_f64
    from synth import make_prompt_states
    z_ref = {}
    for j in which:
        i = sample[j]
        O = states_to_f64(make_prompt_states(wl, lens, requests=[i]), wl.act_fmt)
        cap = {"_only": {"attn"}}
        zi, hi, _ = orc.prefill_one(*O, capture=cap)
        z_ref[j] = zi
        eh = rel_fro(got["hdraft"][j], hi)
        ea = check_attention([got["attn"][j]], [cap["attn"]], fmt, ("request", i))
        say(f"  request {i} (n={int(lens[i])}): h_draft rel err {eh:.3e}, attention rel err {ea:.3e}")
        assert eh <= TOL_HDRAFT[fmt]
    return z_ref


def _sample(lens, *quantiles):
    """Indices of the shortest, the given quantiles and the longest request."""
    order = np.argsort(lens, kind="stable")
    picks = [int(order[0])] + [int(order[int(q * len(order))]) for q in quantiles] + [int(order[-1])]
    return list(dict.fromkeys(picks))


@pytest.mark.timeout(900)
def test_8b_256_request_prefill_in_one_call():
    from oracle import oracle_from_workload
    from synth import make_lengths, make_weights, workload
    wl = workload(2)
    lens = make_lengths(wl)
    sample = _sample(lens, 0.25)
    say(f"case: 8B bf16 256-request batch, B={len(lens)}, T={int(lens.sum())} in one call, oracle on requests {sample} "
        f"(lengths {[int(lens[i]) for i in sample]}; longest request {int(lens.max())})")
    W = make_weights(wl)
    got = _gpu_prefill_sample(wl, W, lens, sample)
    orc = oracle_from_workload(wl, W)
    z_ref = _oracle_check(orc, wl, lens, sample, got, "bf16", range(len(sample)))
    ez = z_errors(got["z"], [z_ref[j] for j in range(len(sample))])
    say(f"  z rel errors {np.round(ez, 5).tolist()}")
    assert ez.max() <= TOL_Z["bf16"]


@pytest.fixture(scope="module")
def batch_70b_e4m3():
    """70B shape with e4m3 weights: the whole 64-request batch in one
    prefill call on the GPU; the sampled requests' outputs kept on the host
    with the oracle built from the same weights."""
    from oracle import oracle_from_workload
    from synth import make_lengths, make_weights, workload
    wl = workload(4)
    lens = make_lengths(wl)
    sample = _sample(lens)
    say(f"case: 70B e4m3 64-request batch, B={len(lens)}, T={int(lens.sum())} in one call, oracle on "
        f"requests {sample} (lengths {[int(lens[i]) for i in sample]}; longest request {int(lens.max())})")
    W = make_weights(wl)
    say("  weights generated")
    got = _gpu_prefill_sample(wl, W, lens, sample)
    orc = oracle_from_workload(wl, W)
    del W
    say("  oracle weights decoded")
    return {"wl": wl, "lens": lens, "sample": sample, "got": got, "orc": orc, "z_ref": {}}


@pytest.mark.timeout(900)
def test_70b_e4m3_batch_shortest_request(batch_70b_e4m3):
    c = batch_70b_e4m3
    c["z_ref"].update(_oracle_check(c["orc"], c["wl"], c["lens"], c["sample"], c["got"], "e4m3", [0]))


@pytest.mark.timeout(900)
def test_70b_e4m3_batch_longest_request(batch_70b_e4m3):
    """The 16,384-token prompt (the configuration's clip): attention over
    256 64-key tiles per query tile, two-block work items."""
    c = batch_70b_e4m3
    last = len(c["sample"]) - 1
    c["z_ref"].update(_oracle_check(c["orc"], c["wl"], c["lens"], c["sample"], c["got"], "e4m3", [last]))
    if 0 not in c["z_ref"]:
        c["z_ref"].update(_oracle_check(c["orc"], c["wl"], c["lens"], c["sample"], c["got"], "e4m3", [0]))
    js = sorted(c["z_ref"])
    ez = z_errors(c["got"]["z"][js], [c["z_ref"][j] for j in js])
    say(f"  z rel errors {np.round(ez, 5).tolist()}")
    assert ez.max() <= TOL_Z["e4m3"]


@pytest.mark.timeout(900)
def test_decode_512_slots_long_caches():
    """512 slots with U[256, 8192] cached tokens: the step's 137k pages cut
    into 256 equal ranges of ~536 pages (one wave per range and KV head),
    walked in pieces of at most 64 pages; three steps; the oracle follows
    the shortest cache, one at the 1/8 quantile and the longest (512 pages,
    over one or two ranges, so a segment boundary can fall inside it)."""
    import torch
    from oracle import oracle_from_workload, states_to_f64
    from synth import make_lengths, make_prompt_states, make_step_states, make_weights, workload
    from paper_2609_01068_amd.predictor import to_device
    wl = workload(3)
    lens = make_lengths(wl)
    B = len(lens)
    sample = _sample(lens, 0.125)
    steps = 3
    say(f"case: 8B bf16 decode, {B} slots, {int(lens.sum())} cached tokens, {steps} steps, oracle on slots "
        f"{sample} (caches {[int(lens[i]) for i in sample]}; longest cache {int(lens.max())})")
    W = make_weights(wl)
    chunk = 48
    max_chunk = max(int(lens[i:i + chunk].sum()) for i in range(0, B, chunk))
    pred = _predictor(wl, W, lens, max_batch_tokens=max_chunk, extra=steps + 16)
    got = {j: None for j in sample}
    for i in range(0, B, chunk):
        idx = list(range(i, min(B, i + chunk)))
        sub = [j for j in idx if j in sample]
        H = mixed_prompt_states(wl, lens[idx], [])
        off = np.concatenate([[0], np.cumsum(lens[idx])])
        # sampled requests use their own host draws (generator index = batch index)
        for j in sub:
            k = idx.index(j)
            S = make_prompt_states(wl, lens, requests=[j])
            for d in range(3):
                H[d][off[k]:off[k + 1]] = to_device(S[d])
        z, hd = pred.prefill(idx, lens[idx], *H, want_hdraft=True)
        rows = [(int(off[idx.index(j)]), int(off[idx.index(j) + 1])) for j in sub]
        att = attention_rows(pred, rows)
        for j, (a, b), at in zip(sub, rows, att):
            got[j] = (float(z[idx.index(j)]), tensor_to_f64(hd[a:b]), at)
        torch.cuda.synchronize()
        say(f"  prefilled slots {idx[0]}..{idx[-1]}")
    orc = oracle_from_workload(wl, W)
    states, z_pre = {}, []
    for j in sample:
        cap = {"_only": {"attn"}}
        zi, hi, st = orc.prefill_one(*states_to_f64(make_prompt_states(wl, lens, requests=[j]), wl.act_fmt),
                                     capture=cap)
        states[j] = st
        z_pre.append(zi)
        eh = rel_fro(got[j][1], hi)
        ea = check_attention([got[j][2]], [cap["attn"]], "bf16", ("prefill", j))
        say(f"  prefill slot {j} (n={int(lens[j])}): h_draft rel err {eh:.3e}, attention rel err {ea:.3e}")
        assert eh <= TOL_HDRAFT["bf16"]
    ez = z_errors([got[j][0] for j in sample], z_pre)
    assert ez.max() <= TOL_Z["bf16"], ez
    slots = list(range(B))
    for t in range(1, steps + 1):
        S = mixed_step_states(wl, B, t, sample)
        z, hd = pred.step(slots, *S, want_hdraft=True)
        zg, hg = tensor_to_f64(z), tensor_to_f64(hd)
        att = attention_rows(pred, [(j, j + 1) for j in sample])
        zr = []
        for j, at in zip(sample, att):
            sj = states_to_f64(make_step_states(wl, B, t, requests=[j]), wl.act_fmt)
            cap = {"_only": {"attn"}}
            zj, hr = orc.step_one(states[j], sj[0][0], sj[1][0], sj[2][0], capture=cap)
            zr.append(zj)
            eh = rel_fro(hg[j], hr)
            ea = check_attention([at], [cap["attn"]], "bf16", ("step", t, j))
            say(f"  step {t} slot {j} (cache {int(lens[j]) + t - 1}): h_draft rel err {eh:.3e}, "
                f"attention rel err {ea:.3e}")
            assert eh <= TOL_HDRAFT["bf16"]
        ez = z_errors(zg[sample], zr)
        say(f"  step {t}: z rel errors {np.round(ez, 5).tolist()}")
        assert ez.max() <= TOL_Z["bf16"]
    pred.close()
