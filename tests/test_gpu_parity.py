"""GPU parity of the HIP path against the fp64 oracle (MI355X, through the C ABI).

Every case prints its name before touching the GPU.  Tolerances: draft
states as relative Frobenius error per request (1e-4 fp32, 2e-2 bf16, 6e-2
e4m3 weights); predicted log-length |dz| <= 1e-2 * max(|z|, rms(z)) (1e-4 for
fp32); integer metadata bit-exact.
"""
import numpy as np
import pytest

from oracle import meta
from gpu_common import (TOL_HDRAFT, TOL_VARIANT, TOL_Z, attention_rows, check_attention, device_states,
                        device_tokens, make_case, make_predictor, oracle_for, oracle_states, reduced_shape,
                        rel_fro, require_gpu, say, step_inputs, step_tokens, tensor_to_f64, z_errors)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _split(arr, lens):
    off = np.concatenate([[0], np.cumsum(lens)])
    return [arr[off[i]:off[i + 1]] for i in range(len(lens))]


def _check_meta(pred, lens, slots, alloc):
    from paper_2609_01068_amd import binding as B
    assert np.array_equal(pred.meta(B.OUTLETS_META_DEV_CU_SEQLENS), meta.cu_seqlens(lens))
    assert np.array_equal(pred.meta(B.OUTLETS_META_DEV_POSITIONS), meta.positions(lens))
    assert np.array_equal(pred.meta(B.OUTLETS_META_DEV_LAST_IDX), meta.last_idx(lens))
    assert np.array_equal(pred.meta(B.OUTLETS_META_DEV_TOKEN_SLOT), np.repeat(slots, lens))
    table = alloc.table().reshape(-1)
    assert np.array_equal(pred.meta(B.OUTLETS_META_PAGE_TABLE), table)
    dev = pred.meta(B.OUTLETS_META_DEV_PAGE_TABLE)
    used = table >= 0
    assert np.array_equal(dev[used], table[used])


def _run_prefill_case(case, keep=True, steps=0, check_intermediates=True):
    fmt = case.fmt
    lens = case.lens
    n = len(lens)
    slots = list(range(n))
    pred = make_predictor(case, keep=keep, max_seq_len=int(lens.max()) + steps + 16)
    H = device_states(case)
    z, hd = pred.prefill(slots, lens, *H, want_hdraft=True, tokens=device_tokens(case.tokens))
    z = tensor_to_f64(z)
    hd = tensor_to_f64(hd)
    orc = oracle_for(case)
    O = oracle_states(case)
    off = np.concatenate([[0], np.cumsum(lens)])
    states, z_ref = [], []
    caps = []
    for i in range(n):
        cap = {}
        tok = None if case.tokens is None else case.tokens[off[i]:off[i + 1]]
        zi, hi, st = orc.prefill_one(*(x[off[i]:off[i + 1]] for x in O), capture=cap, tokens=tok)
        z_ref.append(zi)
        states.append(st)
        caps.append(cap)
        err = rel_fro(hd[off[i]:off[i + 1]], hi)
        assert err <= TOL_HDRAFT[fmt], (i, err)
    ez = z_errors(z, z_ref)
    say(f"  prefill z max rel err {ez.max():.3e}; z_ref rms {np.sqrt(np.mean(np.square(z_ref))):.3e}")
    assert ez.max() <= TOL_Z[fmt], ez
    # the attention output itself, per request (always kept by the library)
    worst = check_attention(attention_rows(pred, [(off[i], off[i + 1]) for i in range(n)]),
                            [c["attn"] for c in caps], fmt, "prefill")
    say(f"  prefill attention worst rel err {worst:.3e}")
    if keep and check_intermediates:
        import torch
        names = [("FUSED", "fused", torch.float32), ("X1", "x1", torch.float32),
                 ("X2", "x2", torch.float32), ("HDRAFT", "hdraft", torch.float32)]
        act = pred.act_dtype
        names += [("NORM_ATTN", "norm_attn", act), ("Q", "q", act), ("ATTN", "attn", act),
                  ("NORM_MLP", "norm_mlp", act), ("MLP_ACT", "mlp_act", act)]
        if case.tokens is not None:
            names.append(("NORM_EMB", "norm_emb", act))
        for buf, key, dt in names:
            g = tensor_to_f64(pred.buffer(buf, dt))
            g = g.reshape(int(lens.sum()), -1)
            worst = max(rel_fro(g[off[i]:off[i + 1]], caps[i][key]) for i in range(n))
            say(f"  {buf:9s} worst rel err {worst:.3e}")
            assert worst <= TOL_HDRAFT[fmt], (buf, worst)
        pooled = tensor_to_f64(pred.buffer("POOLED", torch.float32)).reshape(n, -1)
        for i in range(n):
            assert rel_fro(pooled[i], caps[i]["pooled"]) <= TOL_HDRAFT[fmt]
    alloc = meta.PageAllocator(pred.cfg.num_pages, 16, pred.cfg.max_slots, pred.cfg.max_seq_len)
    assert alloc.prefill(slots, lens) == meta.OK
    _check_meta(pred, lens, np.array(slots), alloc)

    worst_step = 0.0
    for t in range(1, steps + 1):
        S, tk = step_inputs(case, t), step_tokens(case, t)
        zs, hs = pred.step(slots, *device_states(case, S), want_hdraft=True, tokens=device_tokens(tk))
        zs, hs = tensor_to_f64(zs), tensor_to_f64(hs)
        scaps = [{"_only": {"attn"}} for _ in range(n)]
        zr, hr = orc.step(states, *oracle_states(case, S), tokens=tk, captures=scaps)
        for i in range(n):
            assert rel_fro(hs[i], hr[i]) <= TOL_HDRAFT[fmt], (t, i)
        ez = z_errors(zs, zr)
        assert ez.max() <= TOL_Z[fmt], (t, ez)
        # decode attention (split-KV chunks and their merge) against the oracle
        worst_step = max(worst_step, check_attention(attention_rows(pred, [(i, i + 1) for i in range(n)]),
                                                     [c["attn"] for c in scaps], fmt, ("step", t)))
        assert alloc.step(slots) == meta.OK
        from paper_2609_01068_amd import binding as B
        assert np.array_equal(pred.meta(B.OUTLETS_META_PAGE_TABLE), alloc.table().reshape(-1))
        assert np.array_equal(pred.meta(B.OUTLETS_META_SEQ_LEN), alloc.seq_lens())
        assert np.array_equal(pred.meta(B.OUTLETS_META_DEV_POSITIONS), np.asarray(lens) + t - 1)
    say(f"  {steps} decode steps match; step attention worst rel err {worst_step:.3e}")
    pred.close()


def test_tiny_fp32_prefill_intermediates_and_steps():
    say("case: tiny fp32 shape (d=256), 4 requests U[16,64], 8 steps")
    _run_prefill_case(make_case(0), keep=True, steps=8)


def test_bf16_reduced_shape_ragged_tiles_and_steps():
    say("case: bf16 d=512 8q/2kv hd128 F1024, lens [1,17,100,300,33], 3 steps")
    case = make_case(1, lens=[1, 17, 100, 300, 33], shape=reduced_shape(), n_req=5)
    _run_prefill_case(case, keep=True, steps=3)


def test_e4m3_reduced_shape_gqa8_and_steps():
    say("case: e4m3 weights d=512 16q/2kv hd128 F1024, lens [5,64,257,16], 2 steps")
    case = make_case(4, lens=[5, 64, 257, 16], shape=reduced_shape(n_q=16, n_kv=2), n_req=4)
    _run_prefill_case(case, keep=True, steps=2)


def test_bf16_head_dim_64_shape():
    say("case: bf16 d=256 4q/4kv hd64 F512, lens [3,40,90]")
    case = make_case(1, lens=[3, 40, 90], shape=reduced_shape(d=256, n_q=4, n_kv=4, hd=64,
                                                             ffn=512, head_hidden=256), n_req=3)
    _run_prefill_case(case, keep=True, steps=1)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("variant", ["plain", "gated", "embed"])
def test_8b_32_request_batch_sampled_requests(variant):
    """8B shape, the 32-request lognormal batch (also with the Gated Attention
    output gate, and with EAGLE-3 input embeddings over the 128,256-entry
    vocabulary), prefill and one decode step of every request as the
    benchmark runs them; the oracle recomputes a sample that always holds
    the shortest and the longest prompt: h_draft, z and the attention output
    of the prefill and of the step."""
    case = make_case(1, attn_gate=variant == "gated", input_embed=variant == "embed")
    lens = case.lens
    B_ = len(lens)
    order = np.argsort(lens, kind="stable")
    sample = sorted({int(order[0]), int(order[1]), int(order[B_ // 3]), int(order[-1])})
    say(f"case: 8B bf16 32-request batch ({variant}), B={B_}, T={int(lens.sum())}, oracle on requests {sample} "
        f"(lengths {[int(lens[i]) for i in sample]}; longest request {int(lens.max())})")
    pred = make_predictor(case, max_seq_len=int(lens.max()) + 16)
    H = device_states(case)
    slots = list(range(B_))
    z, hd = pred.prefill(slots, lens, *H, want_hdraft=True, tokens=device_tokens(case.tokens))
    z = tensor_to_f64(z)
    assert np.all(np.isfinite(z))
    off = np.concatenate([[0], np.cumsum(lens)])
    attn_pre = attention_rows(pred, [(off[i], off[i + 1]) for i in sample])
    orc = oracle_for(case)
    from synth import make_prompt_states, make_prompt_tokens
    z_ref, states, caps = [], [], []
    for i in sample:
        O = oracle_states(case, make_prompt_states(case.wl, lens, requests=[i]))
        tok = make_prompt_tokens(case.wl, lens, requests=[i]) if case.tokens is not None else None
        cap = {"_only": {"attn"}}
        zi, hi, st = orc.prefill_one(*O, capture=cap, tokens=tok)
        z_ref.append(zi)
        states.append(st)
        caps.append(cap)
        err = rel_fro(tensor_to_f64(hd[off[i]:off[i + 1]]), hi)
        say(f"  request {i} (n={int(lens[i])}) h_draft rel err {err:.3e}")
        assert err <= TOL_HDRAFT["bf16"]
    worst = check_attention(attn_pre, [c["attn"] for c in caps], "bf16", "prefill")
    ez = z_errors(z[sample], z_ref)
    say(f"  sampled prefill: attention worst rel err {worst:.3e}, z worst rel err {ez.max():.3e}")
    assert ez.max() <= TOL_Z["bf16"]
    # one decode step of every request (16-page decode chunks at this batch)
    S, tk = step_inputs(case, 1), step_tokens(case, 1)
    zs, hs = pred.step(slots, *device_states(case, S), want_hdraft=True, tokens=device_tokens(tk))
    zs, hs = tensor_to_f64(zs), tensor_to_f64(hs)
    attn_step = attention_rows(pred, [(i, i + 1) for i in sample])
    OS = oracle_states(case, S)
    zr, scaps = [], []
    for j, i in enumerate(sample):
        cap = {"_only": {"attn"}}
        zi, hi = orc.step_one(states[j], OS[0][i], OS[1][i], OS[2][i],
                              None if tk is None else int(tk[i]), capture=cap)
        zr.append(zi)
        scaps.append(cap)
        assert rel_fro(hs[i], hi) <= TOL_HDRAFT["bf16"], i
    worst = check_attention(attn_step, [c["attn"] for c in scaps], "bf16", "step")
    ez = z_errors(zs[sample], zr)
    say(f"  sampled step: attention worst rel err {worst:.3e}, z worst rel err {ez.max():.3e}")
    assert ez.max() <= TOL_Z["bf16"]
    pred.close()


def test_fused_final_norm_pooling_with_and_without_hdraft():
    """8B shape (d = 4096, the fused final-RMSNorm + pooling path): ragged
    32-row tiles and a 1-token request.  z must not depend on whether the
    caller asks for h_draft (only the requests' last rows are stored then),
    and matches the oracle."""
    lens = [40, 1, 33, 100, 64]
    case = make_case(1, lens=lens, n_req=len(lens))
    say(f"case: 8B bf16, lens {lens}, prefill with and without h_draft")
    pred = make_predictor(case, max_slots=16)
    H = device_states(case)
    z1, hd = pred.prefill(list(range(5)), case.lens, *H, want_hdraft=True)
    z1, hd = tensor_to_f64(z1), tensor_to_f64(hd)
    pred.release(list(range(5)))
    z2, none = pred.prefill(list(range(5, 10)), case.lens, *H)
    assert none is None
    assert np.array_equal(tensor_to_f64(z2), z1)
    orc = oracle_for(case)
    O = oracle_states(case)
    off = np.concatenate([[0], np.cumsum(case.lens)])
    z_ref = []
    for i in range(5):
        zi, hi, _ = orc.prefill_one(*(x[off[i]:off[i + 1]] for x in O))
        z_ref.append(zi)
        assert rel_fro(hd[off[i]:off[i + 1]], hi) <= TOL_HDRAFT["bf16"], i
    ez = z_errors(z1, z_ref)
    say(f"  z max rel err {ez.max():.3e}")
    assert ez.max() <= TOL_Z["bf16"], ez
    pred.close()


def test_qkv_rope_epilogue_matches_split_k_reduce():
    """8B shape: a 100-token request prefilled inside a 3,100-token batch
    (the QKV GEMM has >= 256 tiles: RoPE and the K/V page writes run in its
    epilogue) and alone (the QKV GEMM splits K; its reduce kernel sums the
    fp32 partials and applies RoPE and the page writes).  Its z, h_draft and
    its K/V page contents agree up to the split's summation order."""
    import torch
    from paper_2609_01068_amd import binding as B
    lens = [100, 1500, 1500]
    case = make_case(1, lens=lens, n_req=len(lens))
    say(f"case: 8B bf16, lens {lens} (QKV epilogue) vs request 0 alone (split-K reduce)")
    pred = make_predictor(case, max_slots=4, num_pages=4 * (1600 // 16 + 8))
    H = device_states(case)
    z_all, hd_all = pred.prefill([0, 1, 2], case.lens, *H, want_hdraft=True)
    z_all, hd_all = tensor_to_f64(z_all), tensor_to_f64(hd_all)

    def pages_of(slot, n):
        table = pred.meta(B.OUTLETS_META_PAGE_TABLE).reshape(pred.cfg.max_slots, -1)
        ids = table[slot, :(n + 15) // 16]
        assert np.all(ids >= 0)
        kp = pred.buffer("K_POOL", torch.bfloat16).float().cpu().numpy().reshape(-1, 8, 16, 128)
        vp = pred.buffer("V_POOL", torch.bfloat16).float().cpu().numpy().reshape(-1, 8, 128, 16)
        k = kp[ids].transpose(0, 2, 1, 3).reshape(-1, 8, 128)[:n]          # [token, kv head, ch]
        v = vp[ids].transpose(0, 3, 1, 2).reshape(-1, 8, 128)[:n]
        return k.astype(np.float64), v.astype(np.float64)

    k_all, v_all = pages_of(0, 100)
    z1, hd1 = pred.prefill([3], case.lens[:1], *[x[:100].contiguous() for x in H], want_hdraft=True)
    z1, hd1 = tensor_to_f64(z1), tensor_to_f64(hd1)
    k1, v1 = pages_of(3, 100)
    ek, ev = rel_fro(k_all, k1), rel_fro(v_all, v1)
    eh = rel_fro(hd_all[:100], hd1)
    say(f"  K pages rel err {ek:.2e}, V pages {ev:.2e}, h_draft {eh:.2e}, z {z_all[0]:.6f} vs {z1[0]:.6f}")
    assert ek <= 1e-2 and ev <= 1e-2 and eh <= 1e-2
    assert abs(z_all[0] - z1[0]) <= 1e-2 * max(abs(z1[0]), float(np.sqrt(np.mean(z_all ** 2))))
    pred.close()


def test_packing_and_permutation_invariance():
    say("case: bf16 reduced shape, packed batch vs one-by-one vs permuted")
    case = make_case(1, lens=[7, 130, 1, 64], shape=reduced_shape(), n_req=4)
    lens = case.lens
    pred = make_predictor(case, max_slots=16)
    H = device_states(case)
    z, hd = pred.prefill([0, 1, 2, 3], lens, *H, want_hdraft=True)
    z, hd = tensor_to_f64(z), tensor_to_f64(hd)
    pred.release([0, 1, 2, 3])
    off = np.concatenate([[0], np.cumsum(lens)])
    for i in range(4):
        Hi = [x[off[i]:off[i + 1]].contiguous() for x in H]
        zi, hi = pred.prefill([4 + i], [lens[i]], *Hi, want_hdraft=True)
        assert tensor_to_f64(zi)[0] == z[i]
        assert np.array_equal(tensor_to_f64(hi), hd[off[i]:off[i + 1]])
    pred.release([4, 5, 6, 7])
    perm = [2, 0, 3, 1]
    import torch
    Hp = [torch.cat([x[off[i]:off[i + 1]] for i in perm]) for x in H]
    zp, _ = pred.prefill([8, 9, 10, 11], lens[perm], *Hp, want_hdraft=True)
    assert np.array_equal(tensor_to_f64(zp), z[perm])
    pred.close()


def test_incremental_steps_equal_prefill_recompute():
    say("case: bf16 reduced shape, prefill n then 18 steps vs prefill of n + t")
    import torch
    case = make_case(1, lens=[30, 15], shape=reduced_shape(), n_req=2)
    pred = make_predictor(case, max_slots=8, max_seq_len=128, max_batch_tokens=256)
    lens = case.lens
    H = device_states(case)
    pred.prefill([0, 1], lens, *H)
    rows = [[x[:30] for x in H], [x[30:45] for x in H]]
    for t in range(1, 19):
        S = device_states(case, step_inputs(case, t))
        zs, hs = pred.step([0, 1], *S, want_hdraft=True)
        for i in range(2):
            rows[i] = [torch.cat([rows[i][j], S[j][i:i + 1]]) for j in range(3)]
        if t in (1, 2, 17, 18):
            for i in range(2):
                n = int(lens[i]) + t
                zf, hf = pred.prefill([4 + i], [n], *[r.contiguous() for r in rows[i]], want_hdraft=True)
                pred.release([4 + i])
                a, b = tensor_to_f64(hs[i]), tensor_to_f64(hf[-1])
                assert rel_fro(a, b) <= 1e-2, (t, i)
                assert abs(float(zs[i]) - float(zf[0])) <= 1e-2 * max(abs(float(zf[0])), 0.05)
    pred.close()


@pytest.mark.timeout(600)
def test_step_batch_sizes_across_row_tile_variants():
    """8B shape: a decode step of B requests in one call (B = 64, 65, 200,
    520: the GEMMs run on 64-, 128-, 128- and 256-row tiles, with different
    K splits) equals the same step taken one request per call (1-row calls)
    on a second context with the same weights and history, to the spread of
    fp32 summation order (TOL_VARIANT).  Sampled requests of each batched
    step (both sides of every row-tile boundary) are also checked against
    the oracle: h_draft, z and the attention output."""
    import torch
    n = 520
    case = make_case(1, lens=[8] * n, n_req=n)
    sample = [0, 31, 63, 64, 127, 128, 199, 255, 256, 519]
    say(f"case: 8B bf16, {n} requests of 8 prompt tokens; batched vs one-per-call steps; oracle on {sample}")
    pa = make_predictor(case, max_slots=n, max_seq_len=64)
    pb = make_predictor(case, max_slots=n, max_seq_len=64)
    H = device_states(case)
    slots = list(range(n))
    pa.prefill(slots, case.lens, *H)
    pb.prefill(slots, case.lens, *H)
    orc = oracle_for(case)
    O = oracle_states(case)
    states = {}
    for i in sample:
        _, _, states[i] = orc.prefill_one(*(x[8 * i:8 * i + 8] for x in O))
    for t, b in enumerate((64, 65, 200, 520), start=1):
        S = step_inputs(case, t)
        SD = device_states(case, S)
        za, ha = pa.step(slots[:b], *[x[:b] for x in SD], want_hdraft=True)
        attn_a = attention_rows(pa, [(i, i + 1) for i in sample if i < b])
        zb, hb = [], []
        for i in range(b):
            z1, h1 = pb.step([i], *[x[i:i + 1] for x in SD], want_hdraft=True)
            zb.append(float(z1[0]))
            hb.append(tensor_to_f64(h1[0]))
        za, ha, zb, hb = tensor_to_f64(za), tensor_to_f64(ha), np.array(zb), np.stack(hb)
        eh = max(rel_fro(ha[i], hb[i]) for i in range(b))
        ez = float(z_errors(za, zb).max())
        OS = oracle_states(case, S)
        zr, caps, hr = [], [], []
        for i in sample:
            if i >= b:
                continue
            cap = {"_only": {"attn"}}
            zi, hi = orc.step_one(states[i], OS[0][i], OS[1][i], OS[2][i], capture=cap)
            zr.append(zi)
            caps.append(cap)
            hr.append(rel_fro(ha[i], hi))
        wa = check_attention(attn_a, [c["attn"] for c in caps], "bf16", ("B", b))
        ezr = float(z_errors(za[[i for i in sample if i < b]], zr).max())
        say(f"  B={b}: batched vs one-per-call: h_draft {eh:.2e}, z {ez:.2e}; vs oracle: h_draft "
            f"{max(hr):.2e}, z {ezr:.2e}, attention {wa:.2e}")
        assert eh <= TOL_VARIANT and ez <= TOL_VARIANT, (b, eh, ez)
        assert max(hr) <= TOL_HDRAFT["bf16"] and ezr <= TOL_Z["bf16"], (b, max(hr), ezr)
    pa.close()
    pb.close()


def test_prefill_attention_query_tile_variants_agree():
    """8B shape: two 1,500-token requests prefilled alone (prompts average
    >= 1,024 tokens: 64-query attention work items, two 32-query blocks per
    workgroup) and together with two 1-token requests (average 751: 32-query
    items) give the same attention output, h_draft and z for the long
    requests (a wave's arithmetic for its 32 queries does not depend on how
    many blocks its workgroup holds; the GEMM plans of the two batch sizes
    may differ in fp32 summation order, hence TOL_VARIANT); both variants'
    attention outputs are checked against the oracle."""
    lens_a = [1500, 1500]
    lens_b = [1500, 1500, 1, 1]
    case = make_case(1, lens=lens_b, n_req=len(lens_b))
    say(f"case: 8B bf16, lens {lens_a} (64-query items) vs {lens_b} (32-query items)")
    pa = make_predictor(case, max_slots=4)
    pb = make_predictor(case, max_slots=4)
    H = device_states(case)
    za, ha = pa.prefill([0, 1], lens_a, *[x[:3000].contiguous() for x in H], want_hdraft=True)
    att_a = attention_rows(pa, [(0, 1500), (1500, 3000)])
    zb, hb = pb.prefill([0, 1, 2, 3], lens_b, *H, want_hdraft=True)
    att_b = attention_rows(pb, [(0, 1500), (1500, 3000)])
    ha, hb = tensor_to_f64(ha), tensor_to_f64(hb)[:3000]
    eh = max(rel_fro(ha[:1500], hb[:1500]), rel_fro(ha[1500:], hb[1500:3000]))
    ea = max(rel_fro(att_a[i], att_b[i]) for i in range(2))
    ez = float(z_errors(tensor_to_f64(za), tensor_to_f64(zb)[:2]).max())
    orc = oracle_for(case)
    O = oracle_states(case)
    caps = []
    for i in range(2):
        cap = {"_only": {"attn"}}
        orc.prefill_one(*(x[1500 * i:1500 * (i + 1)] for x in O), capture=cap)
        caps.append(cap)
    wa = check_attention(att_a, [c["attn"] for c in caps], "bf16", "64-query items")
    wb = check_attention(att_b, [c["attn"] for c in caps], "bf16", "32-query items")
    say(f"  variants: attention {ea:.2e}, h_draft {eh:.2e}, z {ez:.2e}; vs oracle: attention {wa:.2e} / {wb:.2e}")
    assert ea <= TOL_VARIANT and eh <= TOL_VARIANT and ez <= TOL_VARIANT
    pa.close()
    pb.close()


def test_constant_token_prompt_at_long_length():
    say("case: 8B bf16 shape, constant-token prompts n=1 and n=4096")
    import torch
    case = make_case(1, lens=[1, 4096], n_req=2)
    pred = make_predictor(case, max_slots=4)
    row = [x[:1] for x in device_states(case)]
    z1, h1 = pred.prefill([0], [1], *row, want_hdraft=True)
    long = [r.expand(4096, -1).contiguous() for r in row]
    z2, h2 = pred.prefill([1], [4096], *long, want_hdraft=True)
    h1, h2 = tensor_to_f64(h1), tensor_to_f64(h2)
    spread = np.abs(h2 - h2[0:1]).max() / np.abs(h2[0]).max()
    say(f"  row spread {spread:.3e}, |z1 - z2| = {abs(float(z1[0]) - float(z2[0])):.3e}")
    assert spread <= 2e-2
    assert rel_fro(h2[-1], h1[0]) <= 2e-2
    assert abs(float(z1[0]) - float(z2[0])) <= 1e-2 * max(abs(float(z1[0])), 0.05)
    pred.close()


def test_error_paths_leave_state_unchanged():
    say("case: error codes on a live context")
    from paper_2609_01068_amd import binding as B
    case = make_case(0, lens=[20, 20])
    pred = make_predictor(case, max_slots=3, num_pages=4, max_seq_len=64)
    H = device_states(case)
    z, _ = pred.prefill([0, 1], [20, 20], *H)   # 2 pages each: pool full
    table = pred.meta(B.OUTLETS_META_PAGE_TABLE)
    codes = []
    for call in (lambda: pred.prefill([0], [5], *[x[:5] for x in H]),
                 lambda: pred.prefill([2], [5], *[x[:5] for x in H]),
                 lambda: pred.prefill([2, 2], [1, 1], *[x[:2] for x in H]),
                 lambda: pred.prefill([2], [0], *[x[:1] for x in H]),
                 lambda: pred.step([2], *[x[:1] for x in H])):
        with pytest.raises(B.OutletsError) as e:
            call()
        codes.append(e.value.rc)
    assert codes == [B.OUTLETS_ERR_SLOT_BUSY, B.OUTLETS_ERR_OUT_OF_PAGES,
                     B.OUTLETS_ERR_INVALID_ARG, B.OUTLETS_ERR_INVALID_ARG, B.OUTLETS_ERR_SLOT_EMPTY]
    assert np.array_equal(pred.meta(B.OUTLETS_META_PAGE_TABLE), table)
    z0, _ = pred.prefill([], [], *H)            # n_req == 0 is a no-op
    pred.release([1])
    z2, _ = pred.prefill([2], [20], *[x[20:40] for x in H])
    assert abs(float(z2[0]) - float(z[1])) <= 1e-5 * max(abs(float(z[1])), 1e-3)
    pred.close()


def test_decode_steps_over_long_caches_merge_segments():
    """Caches of 69, 38 and 3 pages: the step's ~16-page ranges split the
    first request over five ranges (five partial records merged)."""
    say("case: bf16 d=512 8q/2kv hd128, caches of 1100/600/40 tokens (~16-page decode ranges), 3 steps")
    case = make_case(1, lens=[1100, 600, 40], shape=reduced_shape(), n_req=3)
    _run_prefill_case(case, keep=False, steps=3, check_intermediates=False)


DECODE_PLAN_CASES = {
    # every request over four or five ranges
    "long_caches": lambda n: [1030 + (37 * i) % 71 for i in range(n)],
    # several requests inside each range: segments that end mid-piece
    "short_caches": lambda n: [20 + (29 * i) % 41 for i in range(n)],
}


@pytest.mark.parametrize("kind,n_req", [("long_caches", 100), ("short_caches", 300)])
def test_decode_plan_shapes_against_oracle(kind, n_req):
    """bf16 d=512 8q/2kv hd128, two decode steps: the step's pages are cut
    into equal ranges (one wave per range and KV head) whose parts in each
    request are merged by the combine kernel.  The oracle recomputes sampled
    requests: attention output, h_draft and z of every step."""
    lens = DECODE_PLAN_CASES[kind](n_req)
    case = make_case(1, lens=lens, shape=reduced_shape(), n_req=n_req)
    sample = sorted({0, 1, n_req // 2, n_req - 1, int(np.argmax(lens)), int(np.argmin(lens))})
    say(f"case: bf16 reduced shape, {n_req} caches of {min(lens)}..{max(lens)} tokens ({kind}), "
        f"2 steps, oracle on {sample}")
    pred = make_predictor(case, max_seq_len=max(lens) + 16)
    slots = list(range(n_req))
    pred.prefill(slots, case.lens, *device_states(case))
    orc = oracle_for(case)
    O = oracle_states(case)
    off = np.concatenate([[0], np.cumsum(case.lens)])
    states = {}
    for i in sample:
        _, _, states[i] = orc.prefill_one(*(x[off[i]:off[i + 1]] for x in O))
    for t in (1, 2):
        S = step_inputs(case, t)
        zs, hs = pred.step(slots, *device_states(case, S), want_hdraft=True)
        zs, hs = tensor_to_f64(zs), tensor_to_f64(hs)
        got = attention_rows(pred, [(i, i + 1) for i in sample])
        OS = oracle_states(case, S)
        zr, caps = [], []
        for i in sample:
            cap = {"_only": {"attn"}}
            zi, hi = orc.step_one(states[i], OS[0][i], OS[1][i], OS[2][i], capture=cap)
            zr.append(zi)
            caps.append(cap)
            assert rel_fro(hs[i], hi) <= TOL_HDRAFT["bf16"], (t, i)
        wa = check_attention(got, [c["attn"] for c in caps], "bf16", ("step", t))
        ez = float(z_errors(zs[sample], zr).max())
        say(f"  step {t}: attention worst rel err {wa:.3e}, z {ez:.3e}")
        assert ez <= TOL_Z["bf16"]
    pred.close()


def test_decode_steps_8b_shape():
    say("case: 8B bf16 shape, caches of 600/40 tokens, 2 steps")
    case = make_case(1, lens=[600, 40], n_req=2)
    _run_prefill_case(case, keep=False, steps=2, check_intermediates=False)


# ------------------------------------------------------------- Gated Attention

def test_gated_attention_tiny_fp32_intermediates_and_steps():
    say("case: Gated Attention, tiny fp32 shape, 4 requests U[16,64], 8 steps")
    _run_prefill_case(make_case(0, attn_gate=True), keep=True, steps=8)


def test_gated_attention_bf16_reduced_shape_and_steps():
    say("case: Gated Attention, bf16 d=512 8q/2kv hd128, lens [1,17,100,300,33], 3 steps")
    case = make_case(1, lens=[1, 17, 100, 300, 33], shape=reduced_shape(), n_req=5, attn_gate=True)
    _run_prefill_case(case, keep=True, steps=3)


def test_gated_attention_e4m3_reduced_shape_and_steps():
    say("case: Gated Attention, e4m3 weights d=512 16q/2kv hd128, lens [5,64,257,16], 2 steps")
    case = make_case(4, lens=[5, 64, 257, 16], shape=reduced_shape(n_q=16, n_kv=2), n_req=4,
                     attn_gate=True)
    _run_prefill_case(case, keep=True, steps=2)


def test_gated_attention_decode_over_multi_chunk_caches():
    say("case: Gated Attention, bf16 d=512 8q/2kv hd128, caches of 2100/600/40 tokens (256-key chunks), 3 steps")
    case = make_case(1, lens=[2100, 600, 40], shape=reduced_shape(), n_req=3, attn_gate=True)
    _run_prefill_case(case, keep=False, steps=3, check_intermediates=False)


# ------------------------------------------------------------- MLP probe

@pytest.mark.parametrize("cfg", [0, 1], ids=["tiny-fp32", "bf16-reduced"])
def test_mlp_probe_prefill_steps_and_errors(cfg):
    import dataclasses
    from paper_2609_01068_amd import binding as B
    from oracle import probe_from_stored
    from synth import make_probe_weights
    if cfg == 0:
        case = make_case(0)
    else:
        case = make_case(1, lens=[1, 17, 100, 300, 33], shape=reduced_shape(), n_req=5)
    lens = case.lens
    n = len(lens)
    say(f"case: MLP probe on the mid-depth state, cfg {cfg}, lens {list(lens)}, 3 steps")
    PW = make_probe_weights(case.wl)
    W = dict(case.weights)
    W.update({k: v for k, v in PW.items() if k != "_fmt"})
    W["_fmt"] = {**case.weights["_fmt"], **PW["_fmt"]}
    case = dataclasses.replace(case, weights=W)
    pred = make_predictor(case, max_slots=n + 2)
    probe = probe_from_stored(PW)
    H = device_states(case)
    O = oracle_states(case)
    slots = list(range(n))
    off = np.concatenate([[0], np.cumsum(lens)])
    z = tensor_to_f64(pred.probe_prefill(slots, lens, H[1]))
    states, z_ref = [], []
    for i in range(n):
        zi, st = probe.prefill_one(O[1][off[i]:off[i + 1]])
        z_ref.append(zi)
        states.append(st)
    ez = z_errors(z, z_ref)
    say(f"  probe prefill z max rel err {ez.max():.3e}")
    assert ez.max() <= TOL_Z[case.fmt]
    for t in range(1, 4):
        S = step_inputs(case, t)
        zs = tensor_to_f64(pred.probe_step(slots, device_states(case, S)[1]))
        OS = oracle_states(case, S)
        zr = [probe.step_one(states[i], OS[1][i]) for i in range(n)]
        assert z_errors(zs, zr).max() <= TOL_Z[case.fmt], t
    # probe slots are independent of the draft path's slots
    zd, _ = pred.prefill([0], [int(lens[0])], *[x[:int(lens[0])] for x in H])
    codes = []
    for call in (lambda: pred.probe_prefill([0], [1], H[1][:1]),
                 lambda: pred.probe_step([n], H[1][:1]),
                 lambda: pred.probe_prefill([n, n], [1, 1], H[1][:2])):
        with pytest.raises(B.OutletsError) as e:
            call()
        codes.append(e.value.rc)
    assert codes == [B.OUTLETS_ERR_SLOT_BUSY, B.OUTLETS_ERR_SLOT_EMPTY, B.OUTLETS_ERR_INVALID_ARG]
    pred.probe_release(slots + [n])          # inactive slots are a no-op
    z2 = tensor_to_f64(pred.probe_prefill([n], [int(lens[1])], H[1][off[1]:off[2]]))
    assert abs(z2[0] - z[1]) <= 1e-5 * max(abs(z[1]), 1e-3)
    pred.close()


def test_mlp_probe_needs_probe_weights():
    from paper_2609_01068_amd import binding as B
    case = make_case(0, lens=[8])
    pred = make_predictor(case)
    H = device_states(case)
    with pytest.raises(B.OutletsError) as e:
        pred.probe_prefill([0], [8], H[1])
    assert e.value.rc == B.OUTLETS_ERR_UNSUPPORTED
    pred.close()


# ------------------------------------------------------------- draft model head (Eq. 2)

def _with_lm(case):
    import dataclasses
    from synth import make_lm_weights
    LW = make_lm_weights(case.wl)
    W = dict(case.weights)
    W["w_lm"] = LW["w_lm"]
    W["_fmt"] = {**case.weights["_fmt"], **LW["_fmt"]}
    return dataclasses.replace(case, weights=W)


def _check_distribution(p_gpu, h_last, w_lm, fmt, label):
    from oracle import draft_distribution
    ref = draft_distribution(h_last[None, :], w_lm)[0]
    err = rel_fro(p_gpu, ref)
    assert abs(p_gpu.sum() - 1.0) <= 1e-4, label
    assert err <= TOL_HDRAFT[fmt], (label, err)
    return err


@pytest.mark.parametrize("cfg", [0, 1, 4], ids=["tiny-fp32", "bf16-reduced", "e4m3-reduced"])
def test_draft_head_prefill_and_steps(cfg):
    from paper_2609_01068_amd import binding as B
    from oracle.formats import decode_weight
    if cfg == 0:
        case = make_case(0)
    elif cfg == 1:
        case = make_case(1, lens=[1, 17, 100, 300, 33], shape=reduced_shape(), n_req=5)
    else:
        case = make_case(4, lens=[5, 64, 257, 16], shape=reduced_shape(n_q=16, n_kv=2), n_req=4)
    case = _with_lm(case)
    lens = case.lens
    n = len(lens)
    say(f"case: draft model head (V={case.wl.shape.vocab}), cfg {cfg}, lens {list(lens)}, 2 steps")
    pred = make_predictor(case, max_seq_len=int(lens.max()) + 8)
    H = device_states(case)
    slots = list(range(n))
    pred.prefill(slots, lens, *H)
    p = tensor_to_f64(pred.draft_distribution(n))
    orc = oracle_for(case)
    w_lm = decode_weight(case.weights["w_lm"], case.weights["_fmt"]["w_lm"])
    O = oracle_states(case)
    off = np.concatenate([[0], np.cumsum(lens)])
    states, worst = [], 0.0
    for i in range(n):
        _, hi, st = orc.prefill_one(*(x[off[i]:off[i + 1]] for x in O))
        states.append(st)
        worst = max(worst, _check_distribution(p[i], hi[-1], w_lm, case.fmt, ("prefill", i)))
    for t in range(1, 3):
        S = step_inputs(case, t)
        pred.step(slots, *device_states(case, S))
        p = tensor_to_f64(pred.draft_distribution(n))
        _, hr = orc.step(states, *oracle_states(case, S))
        for i in range(n):
            worst = max(worst, _check_distribution(p[i], hr[i], w_lm, case.fmt, ("step", t, i)))
    say(f"  worst distribution rel err {worst:.3e}")
    with pytest.raises(B.OutletsError) as e:
        pred.draft_distribution(n - 1 if n > 1 else 2)
    assert e.value.rc == B.OUTLETS_ERR_INVALID_ARG
    pred.close()


def test_draft_head_absent_without_vocab():
    from paper_2609_01068_amd import binding as B
    case = make_case(0, lens=[8])
    pred = make_predictor(case)
    H = device_states(case)
    pred.prefill([0], [8], *H)
    with pytest.raises(B.OutletsError) as e:
        pred.draft_distribution(1)
    assert e.value.rc == B.OUTLETS_ERR_UNSUPPORTED
    pred.close()


def test_8b_32_request_batch_draft_head_sampled_requests():
    """Eq. 2 at the 8B shape (V = 128,256) on the 32-request batch; the oracle
    recomputes two sampled requests."""
    from oracle.formats import decode_weight
    from synth import make_prompt_states
    case = _with_lm(make_case(1))
    lens = case.lens
    say(f"case: 32-request 8B batch, draft model head, V={case.wl.shape.vocab}, B={len(lens)}, T={int(lens.sum())}")
    pred = make_predictor(case)
    H = device_states(case)
    pred.prefill(list(range(len(lens))), lens, *H)
    p = tensor_to_f64(pred.draft_distribution(len(lens)))
    assert np.all(np.isfinite(p))
    assert np.allclose(p.sum(axis=1), 1.0, atol=1e-4)
    order = np.argsort(lens)
    sample = [int(order[0]), int(order[len(order) // 3])]
    orc = oracle_for(case)
    w_lm = decode_weight(case.weights["w_lm"], case.weights["_fmt"]["w_lm"])
    O = oracle_states(case, make_prompt_states(case.wl, lens, requests=sample))
    o_off = 0
    for i in sample:
        n = int(lens[i])
        _, hi, _ = orc.prefill_one(*(x[o_off:o_off + n] for x in O))
        o_off += n
        err = _check_distribution(p[i], hi[-1], w_lm, "bf16", ("request", i))
        say(f"  request {i} (n={n}) distribution rel err {err:.3e}")
    pred.close()


# ------------------------------------------------------------- input embeddings

def test_input_embeddings_tiny_fp32_intermediates_and_steps():
    say("case: input embeddings, tiny fp32 shape (V=512), 4 requests U[16,64], 6 steps")
    _run_prefill_case(make_case(0, input_embed=True), keep=True, steps=6)


def test_input_embeddings_bf16_reduced_shape_and_steps():
    say("case: input embeddings, bf16 d=512 8q/2kv hd128 V=1024, lens [1,17,100,300,33], 3 steps")
    case = make_case(1, lens=[1, 17, 100, 300, 33], shape=reduced_shape(), n_req=5, input_embed=True)
    _run_prefill_case(case, keep=True, steps=3)


def test_input_embeddings_e4m3_gated_reduced_shape_and_steps():
    say("case: input embeddings + Gated Attention, e4m3 weights d=512 16q/2kv hd128, lens [5,64,257,16], 2 steps")
    case = make_case(4, lens=[5, 64, 257, 16], shape=reduced_shape(n_q=16, n_kv=2), n_req=4,
                     attn_gate=True, input_embed=True)
    _run_prefill_case(case, keep=True, steps=2)


def test_input_embeddings_odd_width_scalar_path():
    say("case: input embeddings, bf16 d=256 4q/4kv hd64 (non-vector gather), lens [3,40,90], 1 step")
    case = make_case(1, lens=[3, 40, 90], shape=reduced_shape(d=256, n_q=4, n_kv=4, hd=64, ffn=512,
                                                             head_hidden=256), n_req=3, input_embed=True)
    _run_prefill_case(case, keep=True, steps=1)


def test_input_embeddings_out_of_range_ids_read_a_zero_row():
    """Ids outside [0, V) cannot be reported from the device: they take a zero
    embedding row (checked against the oracle with an appended zero row)."""
    import torch
    case = make_case(1, lens=[7, 20], shape=reduced_shape(), n_req=2, input_embed=True)
    V = case.wl.shape.vocab
    tok = case.tokens.copy()
    tok[[0, 3, 9, 26]] = [-1, V, -(2 ** 31), 2 ** 31 - 1]
    say(f"case: input embeddings with out-of-range ids {tok[[0, 3, 9, 26]].tolist()}, V={V}")
    pred = make_predictor(case, keep=True)
    z, hd = pred.prefill([0, 1], case.lens, *device_states(case), want_hdraft=True, tokens=device_tokens(tok))
    hd, z = tensor_to_f64(hd), tensor_to_f64(z)
    e = tensor_to_f64(pred.buffer("NORM_EMB", torch.bfloat16)).reshape(len(tok), -1)
    assert np.all(e[[0, 3, 9, 26]] == 0.0)
    orc = oracle_for(case)
    orc.w["embed"] = np.vstack([orc.w["embed"], np.zeros((1, case.wl.shape.d))])
    ref_tok = np.where((tok < 0) | (tok >= V), V, tok)
    O = oracle_states(case)
    zr, hr, _ = orc.prefill(case.lens, *O, tokens=ref_tok)
    for i, (a, b) in enumerate([(0, 7), (7, 27)]):
        assert rel_fro(hd[a:b], hr[a:b]) <= TOL_HDRAFT["bf16"], i
    assert z_errors(z, zr).max() <= TOL_Z["bf16"]
    pred.close()


def test_input_embeddings_need_token_ids_and_weights():
    from paper_2609_01068_amd import binding as B
    case = make_case(1, lens=[4], shape=reduced_shape(), n_req=1, input_embed=True)
    say("case: input-embedding argument errors")
    pred = make_predictor(case)
    H = device_states(case)
    with pytest.raises(B.OutletsError) as ei:
        pred.prefill([0], case.lens, *H)                   # no token ids
    assert ei.value.rc == B.OUTLETS_ERR_INVALID_ARG
    z, _ = pred.prefill([0], case.lens, *H, tokens=device_tokens(case.tokens))   # state unchanged
    assert np.isfinite(tensor_to_f64(z)).all()
    pred.close()
    W = dict(case.weights)
    W.pop("gamma_emb")
    bad = make_case(1, lens=[4], shape=reduced_shape(), n_req=1, input_embed=True)
    bad.weights = W
    with pytest.raises(B.OutletsError) as ei:
        make_predictor(bad)
    assert ei.value.rc == B.OUTLETS_ERR_INVALID_ARG


# ------------------------------------------------------------- e4m3 weight decoding


def test_e4m3_gemm_decodes_all_256_codes_exactly():
    """Every OCP e4m3 code through the e4m3-weight GEMM, bit for bit: the
    fused projection's W_proj holds the 256 codes (twice, in three
    differently shifted columns, one per state tensor), its row scales are
    1.0, and each token's states are one-hot on one of those columns, so the
    fp32 FUSED row is that column's decoded codes (0 * NaN makes a row with
    a NaN code NaN for every token).  Compared exactly with the oracle's
    decode (fp64, exact for every e4m3 value) on a 600-token prefill
    (256-row tiles and a ragged tail) and on a 3-request decode step (the
    small-M split-K path)."""
    import dataclasses
    import torch
    from oracle import decode_weight, fuse
    d = 512
    case = make_case(4, lens=[200, 250, 150], shape=reduced_shape(), n_req=3)
    cols = [5, d + 300, 2 * d + 511]                 # one hot column in each of h_low, h_mid, h_high
    codes = np.zeros((d, 3 * d), dtype=np.uint8)
    for j, (c, shift) in enumerate(zip(cols, (0, 85, 170))):
        codes[:, c] = (np.arange(d) + shift) % 256
    W = dict(case.weights)
    W["w_proj"] = (codes, np.full(d, 0x3F80, dtype=np.uint16))   # bf16 1.0 row scales
    case = dataclasses.replace(case, weights=W)
    w_ref = decode_weight(W["w_proj"], "e4m3")
    say("case: e4m3 GEMM, all 256 codes in W_proj, one-hot states, unit scales; prefill of 600 tokens + 1 step")

    def one_hot(rows, hot):
        X = np.zeros((rows, 3 * d))
        X[np.arange(rows), hot] = 1.0
        bits = (X.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)     # exact in bf16
        return X, [np.ascontiguousarray(bits[:, s * d:(s + 1) * d]) for s in range(3)]

    def check(pred, X, label):
        got = tensor_to_f64(pred.buffer("FUSED", torch.float32)).reshape(X.shape[0], d)
        ref = fuse(w_ref, X[:, :d], X[:, d:2 * d], X[:, 2 * d:])
        assert np.array_equal(np.isnan(got), np.isnan(ref)), label
        assert np.array_equal(got, ref, equal_nan=True), label
        # every finite code is read somewhere outside the NaN rows
        ok = ~np.isnan(ref).any(axis=0)
        seen = set()
        for r, c in enumerate(np.asarray(X).argmax(axis=1)):
            seen.update(int(v) for v in codes[ok, c])
        assert seen >= set(range(256)) - {0x7F, 0xFF}, label
        assert np.isnan(ref[:, codes[:, cols[0]] == 0x7F]).all()
        return int(np.isnan(ref).any(axis=0).sum())

    pred = make_predictor(case, keep=True, max_seq_len=300)
    T = int(case.lens.sum())
    X, S = one_hot(T, [cols[r % 3] for r in range(T)])
    pred.prefill([0, 1, 2], case.lens, *device_states(case, S))
    nan_rows = check(pred, X, "prefill")
    Xs, Ss = one_hot(3, cols)
    pred.step([0, 1, 2], *device_states(case, Ss))
    check(pred, Xs, "step")
    say(f"  FUSED bit-exact vs decoded codes on {T} + 3 rows ({nan_rows} NaN output rows from the NaN codes)")
    pred.close()
