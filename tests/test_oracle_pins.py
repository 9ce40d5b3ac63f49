"""Pins of the fp64 oracle against things other than itself (CPU only).

Each test checks the oracle against a library routine that computes the same
textbook operation, a closed form, an invariant the paper's definitions
imply, or a scalar brute force written from those definitions.  The
mutation tests at the end plant plausible mistakes in the oracle and check
that at least one pin fails.
"""
import math

import numpy as np
import pytest
import torch

import oracle.model as oracle_model
from oracle import (OracleModel, OracleShape, causal_gqa_attention, decode_bf16,
                    decode_e4m3, fuse, length_head, rms_norm, rope, silu)

TINY = OracleShape(d=8, n_q=2, n_kv=1, head_dim=4, ffn=12, head_hidden=6, rope_theta=1e4)
SMALL = OracleShape(d=32, n_q=4, n_kv=2, head_dim=8, ffn=40, head_hidden=16, rope_theta=1e4)


def rand_weights(shape: OracleShape, seed=0, scale=0.3):
    r = np.random.default_rng(seed)
    d, hd = shape.d, shape.head_dim
    g = lambda *s: r.standard_normal(s) * scale  # noqa: E731
    return {
        "w_proj": g(d, 3 * d), "w_q": g(shape.n_q * hd, d), "w_k": g(shape.n_kv * hd, d),
        "w_v": g(shape.n_kv * hd, d), "w_o": g(d, shape.n_q * hd),
        "w_gate": g(shape.ffn, d), "w_up": g(shape.ffn, d), "w_down": g(d, shape.ffn),
        "gamma_attn": 1 + g(d), "gamma_mlp": 1 + g(d), "gamma_final": 1 + g(d),
        "head_w1": g(shape.head_hidden, 2 * d), "head_b1": g(shape.head_hidden),
        "head_w2": g(shape.head_hidden), "head_b2": g(1),
    }


def rand_states(n, d, seed):
    r = np.random.default_rng(seed)
    return [r.standard_normal((n, d)) * s for s in (1.0, 2.0, 4.0)]


# ------------------------------------------------------------- formats

def test_e4m3_all_codes_match_torch_float8():
    codes = np.arange(256, dtype=np.uint8)
    ours = decode_e4m3(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(ours[ok], ref[ok])
    assert np.isnan(ours).sum() == 2          # S.1111.111 only


def test_e4m3_spec_values():
    # OCP OFP8 E4M3: max normal 448, min normal 2^-6, min subnormal 2^-9, 1.0 = 0x38
    known = {0x7E: 448.0, 0xFE: -448.0, 0x08: 2.0 ** -6, 0x01: 2.0 ** -9, 0x38: 1.0,
             0x00: 0.0, 0x07: 7 * 2.0 ** -9, 0x40: 2.0, 0xB8: -1.0, 0x3C: 1.5}
    got = decode_e4m3(np.array(list(known), dtype=np.uint8))
    assert np.array_equal(got, np.array(list(known.values())))


def test_bf16_decode_matches_torch():
    bits = np.random.default_rng(1).integers(0, 2 ** 16, size=4096).astype(np.uint16)
    bits = bits[(bits & 0x7F80) != 0x7F80]     # drop inf/nan patterns
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(decode_bf16(bits), ref)
    assert decode_bf16(np.array([0x3F80, 0xC000], np.uint16)).tolist() == [1.0, -2.0]


# ------------------------------------------------------------- elementwise / norms

def test_rms_norm_matches_torch():
    r = np.random.default_rng(2)
    x, g = r.standard_normal((7, 33)) * 3, r.standard_normal(33)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (33,), torch.from_numpy(g), eps=1e-5)
    assert np.allclose(rms_norm(x, g, 1e-5), ref.numpy(), rtol=1e-13, atol=1e-13)


def test_rms_norm_scale_invariant_as_eps_vanishes():
    r = np.random.default_rng(3)
    x, g = r.standard_normal((4, 16)), r.standard_normal(16)
    assert np.allclose(rms_norm(37.5 * x, g, 0.0), rms_norm(x, g, 0.0), rtol=1e-13)
    # unit gamma: every row has unit root-mean-square
    y = rms_norm(x, np.ones(16), 0.0)
    assert np.allclose(np.sqrt((y * y).mean(axis=1)), 1.0, rtol=1e-13)


def test_silu_matches_torch():
    u = np.linspace(-30, 30, 1001)
    assert np.allclose(silu(u), torch.nn.functional.silu(torch.from_numpy(u)).numpy(),
                       rtol=1e-14, atol=1e-300)


# ------------------------------------------------------------- rotary

def test_rope_position_zero_is_identity():
    x = np.random.default_rng(4).standard_normal((1, 3, 16))
    assert np.array_equal(rope(x, np.array([0]), 1e4), x)


def test_rope_is_complex_rotation():
    _check_rope_complex(rope)


def _check_rope_complex(rope_fn):
    # pair (c, c + hd/2) as the complex number x_c + i x_{c+hd/2}, rotated by e^{i p w_c}
    hd, theta = 16, 5e5
    r = np.random.default_rng(5)
    x = r.standard_normal((6, 2, hd))
    pos = np.array([0, 1, 7, 100, 4095, 16383])
    z = x[..., :hd // 2] + 1j * x[..., hd // 2:]
    w = np.array([theta ** (-(2 * c) / hd) for c in range(hd // 2)])
    zr = z * np.exp(1j * pos[:, None, None] * w[None, None, :])
    ref = np.concatenate([zr.real, zr.imag], axis=-1)
    assert np.allclose(rope_fn(x, pos, theta), ref, rtol=1e-12, atol=1e-12)


def test_rope_preserves_norm_and_relative_position():
    r = np.random.default_rng(6)
    q, k = r.standard_normal((1, 1, 8)), r.standard_normal((1, 1, 8))
    assert np.isclose(np.linalg.norm(rope(q, np.array([123]), 1e4)), np.linalg.norm(q))
    s1 = (rope(q, np.array([10]), 1e4) * rope(k, np.array([3]), 1e4)).sum()
    s2 = (rope(q, np.array([510]), 1e4) * rope(k, np.array([503]), 1e4)).sum()
    assert np.isclose(s1, s2, rtol=1e-10)


# ------------------------------------------------------------- attention

def _sdpa_ref(q, k, v, causal):
    group = q.shape[1] // k.shape[1]
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    kt = torch.from_numpy(k).repeat_interleave(group, dim=1).permute(1, 0, 2)[None]
    vt = torch.from_numpy(v).repeat_interleave(group, dim=1).permute(1, 0, 2)[None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=causal)
    return o[0].permute(1, 0, 2).numpy()


def test_prefill_attention_matches_torch_sdpa():
    _check_sdpa(causal_gqa_attention)


def _check_sdpa(attn):
    r = np.random.default_rng(7)
    n, hq, hkv, hd = 37, 8, 2, 16
    q, k, v = r.standard_normal((n, hq, hd)), r.standard_normal((n, hkv, hd)), r.standard_normal((n, hkv, hd))
    pos = np.arange(n)
    got = attn(q, k, v, pos, pos, chunk=10)
    assert np.allclose(got, _sdpa_ref(q, k, v, True), rtol=1e-12, atol=1e-12)


def test_decode_attention_matches_torch_sdpa():
    r = np.random.default_rng(8)
    n, hq, hkv, hd = 29, 4, 1, 8
    q, k, v = r.standard_normal((1, hq, hd)), r.standard_normal((n, hkv, hd)), r.standard_normal((n, hkv, hd))
    got = causal_gqa_attention(q, k, v, np.array([n - 1]), np.arange(n))
    assert np.allclose(got, _sdpa_ref(q, k, v, False), rtol=1e-12, atol=1e-12)


def test_one_token_attention_returns_its_value_row():
    _check_one_token(causal_gqa_attention)


# ------------------------------------------------------------- fusion / head

def test_fusion_is_blockwise_linear_in_low_mid_high_order():
    r = np.random.default_rng(10)
    d = 6
    w = r.standard_normal((d, 3 * d))
    hl, hm, hh = r.standard_normal((4, d)), r.standard_normal((4, d)), r.standard_normal((4, d))
    ref = hl @ w[:, :d].T + hm @ w[:, d:2 * d].T + hh @ w[:, 2 * d:].T
    assert np.allclose(fuse(w, hl, hm, hh), ref, rtol=1e-13, atol=1e-13)


def test_head_relu_cut_and_linear_branch():
    r = np.random.default_rng(11)
    p = r.standard_normal((3, 10))
    w1, w2 = r.standard_normal((5, 10)), r.standard_normal(5)
    # every hidden unit off -> output is the final bias
    assert np.allclose(length_head(p, w1, np.full(5, -1e6), w2, np.array([0.25])), 0.25)
    # every hidden unit on -> plain affine map
    z = length_head(p, w1, np.full(5, 1e6), w2, np.array([0.0]))
    assert np.allclose(z, (p @ w1.T + 1e6) @ w2, rtol=1e-12)


# ------------------------------------------------------------- scalar brute force

def _brute_prefill(shape, W, hl, hm, hh):
    """The whole layer + head with scalar loops and the math module only."""
    n, d, hd, hq, hkv = len(hl), shape.d, shape.head_dim, shape.n_q, shape.n_kv
    eps = shape.rms_eps

    def mv(mat, vec):
        return [sum(mat[i][j] * vec[j] for j in range(len(vec))) for i in range(len(mat))]

    def norm(vec, g):
        rms = math.sqrt(sum(t * t for t in vec) / len(vec) + eps)
        return [vec[i] / rms * g[i] for i in range(len(vec))]

    def rot(vec, p):
        h2 = hd // 2
        out = list(vec)
        for c in range(h2):
            ang = p * shape.rope_theta ** (-2.0 * c / hd)
            out[c] = vec[c] * math.cos(ang) - vec[c + h2] * math.sin(ang)
            out[c + h2] = vec[c + h2] * math.cos(ang) + vec[c] * math.sin(ang)
        return out

    Wl = {k: np.asarray(v).tolist() for k, v in W.items()}
    F, Q, K, V = [], [], [], []
    for t in range(n):
        x = list(hl[t]) + list(hm[t]) + list(hh[t])
        f = mv(Wl["w_proj"], x)
        a = norm(f, Wl["gamma_attn"])
        q, k, v = mv(Wl["w_q"], a), mv(Wl["w_k"], a), mv(Wl["w_v"], a)
        Q.append([rot(q[h * hd:(h + 1) * hd], t) for h in range(hq)])
        K.append([rot(k[h * hd:(h + 1) * hd], t) for h in range(hkv)])
        V.append([v[h * hd:(h + 1) * hd] for h in range(hkv)])
        F.append(f)
    Hd = []
    for t in range(n):
        o = []
        for h in range(hq):
            g = h // (hq // hkv)
            s = [sum(Q[t][h][c] * K[j][g][c] for c in range(hd)) / math.sqrt(hd) for j in range(t + 1)]
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            tot = sum(e)
            o += [sum(e[j] / tot * V[j][g][c] for j in range(t + 1)) for c in range(hd)]
        x1 = [F[t][i] + y for i, y in enumerate(mv(Wl["w_o"], o))]
        b = norm(x1, Wl["gamma_mlp"])
        gt, up = mv(Wl["w_gate"], b), mv(Wl["w_up"], b)
        m = [gt[i] / (1 + math.exp(-gt[i])) * up[i] for i in range(len(gt))]
        x2 = [x1[i] + y for i, y in enumerate(mv(Wl["w_down"], m))]
        Hd.append(norm(x2, Wl["gamma_final"]))
    pooled = [sum(Hd[t][i] for t in range(n)) / n for i in range(d)] + Hd[n - 1]
    u = [max(0.0, y + Wl["head_b1"][i]) for i, y in enumerate(mv(Wl["head_w1"], pooled))]
    z = sum(u[i] * Wl["head_w2"][i] for i in range(len(u))) + Wl["head_b2"][0]
    return z, np.array(Hd)


@pytest.mark.parametrize("n", [1, 2, 5])
def test_prefill_matches_scalar_brute_force(n):
    _check_brute(OracleModel, n)


def _check_brute(model_cls, n):
    W = rand_weights(TINY, seed=12)
    hl, hm, hh = rand_states(n, TINY.d, seed=13 + n)
    z, hd, _ = model_cls(TINY, W).prefill_one(hl, hm, hh)
    zb, hb = _brute_prefill(TINY, W, hl, hm, hh)
    assert abs(z - zb) < 1e-11
    assert np.allclose(hd, hb, rtol=1e-11, atol=1e-11)


# ------------------------------------------------------------- pipeline invariants

def test_constant_token_prompt_gives_length_independent_prediction():
    W = rand_weights(SMALL, seed=14)
    m = OracleModel(SMALL, W)
    row = rand_states(1, SMALL.d, seed=15)
    zs = []
    for n in (1, 5, 17):
        z, hd, _ = m.prefill_one(*[np.repeat(x, n, axis=0) for x in row])
        assert np.allclose(hd, hd[0:1], rtol=1e-12, atol=1e-12)
        zs.append(z)
    assert np.allclose(zs, zs[0], rtol=1e-12, atol=1e-12)


def test_incremental_steps_equal_prefill_recompute():
    W = rand_weights(SMALL, seed=16)
    m = OracleModel(SMALL, W)
    n, t_max = 9, 4
    hl, hm, hh = rand_states(n + t_max, SMALL.d, seed=17)
    _, _, st = m.prefill_one(hl[:n], hm[:n], hh[:n])
    for t in range(1, t_max + 1):
        z_step, h_step = m.step_one(st, hl[n + t - 1], hm[n + t - 1], hh[n + t - 1])
        z_full, h_full, _ = m.prefill_one(hl[:n + t], hm[:n + t], hh[:n + t])
        assert abs(z_step - z_full) < 1e-12
        assert np.allclose(h_step, h_full[-1], rtol=1e-11, atol=1e-12)


def test_zero_inputs_closed_form():
    W = rand_weights(SMALL, seed=18)
    z, hd, _ = OracleModel(SMALL, W).prefill_one(*[np.zeros((6, SMALL.d))] * 3)
    assert np.array_equal(hd, np.zeros_like(hd))
    ref = np.maximum(W["head_b1"], 0) @ W["head_w2"] + W["head_b2"][0]
    assert abs(z - ref) < 1e-15


def test_causal_prefix_is_unaffected_by_later_tokens():
    W = rand_weights(SMALL, seed=19)
    m = OracleModel(SMALL, W)
    a = rand_states(8, SMALL.d, seed=20)
    b = [x.copy() for x in a]
    for x in b:
        x[5:] = np.random.default_rng(21).standard_normal(x[5:].shape)
    _, ha, _ = m.prefill_one(*a)
    _, hb, _ = m.prefill_one(*b)
    assert np.allclose(ha[:5], hb[:5], rtol=1e-13, atol=1e-13)
    assert not np.allclose(ha[5:], hb[5:])


def test_packing_and_permutation():
    W = rand_weights(SMALL, seed=22)
    m = OracleModel(SMALL, W)
    lens = [3, 7, 1, 5]
    per = [rand_states(n, SMALL.d, seed=30 + i) for i, n in enumerate(lens)]
    packed = [np.concatenate([p[j] for p in per]) for j in range(3)]
    z, hd, _ = m.prefill(lens, *packed)
    perm = [2, 0, 3, 1]
    packed_p = [np.concatenate([per[i][j] for i in perm]) for j in range(3)]
    zp, hdp, _ = m.prefill([lens[i] for i in perm], *packed_p)
    assert np.array_equal(zp, z[perm])
    off = np.concatenate([[0], np.cumsum(lens)])
    offp = np.concatenate([[0], np.cumsum([lens[i] for i in perm])])
    for k, i in enumerate(perm):
        assert np.array_equal(hdp[offp[k]:offp[k + 1]], hd[off[i]:off[i + 1]])


# ------------------------------------------------------------- gated attention

def _gated_model(seed=11, zero_gate=False):
    W = rand_weights(SMALL, seed=seed)
    r = np.random.default_rng(seed + 1)
    W["w_attn_gate"] = (np.zeros((SMALL.n_q * SMALL.head_dim, SMALL.d)) if zero_gate
                        else r.standard_normal((SMALL.n_q * SMALL.head_dim, SMALL.d)) * 0.3)
    return W


def test_zero_gate_weights_halve_the_attention_output():
    # sigmoid(0) = 1/2 exactly: the gated output is half the plain one
    hl, hm, hh = rand_states(9, SMALL.d, 3)
    W = _gated_model(zero_gate=True)
    plain = {k: v for k, v in W.items() if k != "w_attn_gate"}
    cg, cp = {}, {}
    OracleModel(SMALL, W).prefill_one(hl, hm, hh, capture=cg)
    OracleModel(SMALL, plain).prefill_one(hl, hm, hh, capture=cp)
    assert np.array_equal(cg["attn"], 0.5 * cp["attn"])


def _check_gated_layer():
    # torch fp64 SDPA on the oracle's roped q/k/v, times torch.sigmoid of the
    # gate projection of the normed input, must equal the oracle's output
    n = 13
    hl, hm, hh = rand_states(n, SMALL.d, 4)
    W = _gated_model()
    cap = {}
    OracleModel(SMALL, W).prefill_one(hl, hm, hh, capture=cap)
    q = cap["q"].reshape(n, SMALL.n_q, SMALL.head_dim)
    o = _sdpa_ref(q, cap["k"], cap["v"], True).reshape(n, -1)
    gate = torch.sigmoid(torch.from_numpy(cap["norm_attn"]) @ torch.from_numpy(W["w_attn_gate"]).T).numpy()
    assert np.allclose(cap["attn"], o * gate, rtol=1e-12, atol=1e-12)


def test_gated_attention_matches_torch_sdpa_times_sigmoid_gate():
    _check_gated_layer()


def test_gate_is_absent_without_gate_weights():
    hl, hm, hh = rand_states(6, SMALL.d, 5)
    W = rand_weights(SMALL, seed=12)
    cap = {}
    OracleModel(SMALL, W).prefill_one(hl, hm, hh, capture=cap)
    q = cap["q"].reshape(6, SMALL.n_q, SMALL.head_dim)
    assert np.allclose(cap["attn"], _sdpa_ref(q, cap["k"], cap["v"], True).reshape(6, -1),
                       rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------- input embeddings

VOCAB = 23


def _embed_model(seed=41, gated=False):
    """SMALL model with EAGLE-3 input embeddings: Q/K/V (and gate) over 2d."""
    W = _gated_model(seed) if gated else rand_weights(SMALL, seed=seed)
    r = np.random.default_rng(seed + 1)
    for k in ("w_q", "w_k", "w_v") + (("w_attn_gate",) if gated else ()):
        W[k] = np.concatenate([r.standard_normal(W[k].shape) * 0.3, W[k]], axis=1)
    W["embed"] = r.standard_normal((VOCAB, SMALL.d)) * 0.5
    W["gamma_emb"] = 1 + r.standard_normal(SMALL.d) * 0.3
    return W


def _check_embed_layer(gated=False):
    # torch's own rms_norm of the gathered embedding rows and of f_ctx,
    # concatenated embedding-first, must give the oracle's values (v has no
    # RoPE; q at position 0 is unrotated) and, when gated, its gate input
    import torch.nn.functional as F
    n = 11
    hl, hm, hh = rand_states(n, SMALL.d, 42)
    tok = np.random.default_rng(43).integers(0, VOCAB, n)
    W = _embed_model(gated=gated)
    cap = {}
    OracleModel(SMALL, W).prefill_one(hl, hm, hh, capture=cap, tokens=tok)
    t = torch.from_numpy
    e = F.rms_norm(t(W["embed"])[t(tok)], (SMALL.d,), t(W["gamma_emb"]), SMALL.rms_eps)
    a = F.rms_norm(t(cap["fused"]), (SMALL.d,), t(W["gamma_attn"]), SMALL.rms_eps)
    x = torch.cat([e, a], dim=1)
    assert np.allclose(cap["norm_emb"], e.numpy(), rtol=1e-12, atol=1e-12)
    v = (x @ t(W["w_v"]).T).reshape(n, SMALL.n_kv, SMALL.head_dim).numpy()
    assert np.allclose(cap["v"], v, rtol=1e-12, atol=1e-12)
    q0 = (x[:1] @ t(W["w_q"]).T).numpy()
    assert np.allclose(cap["q"][:1], q0, rtol=1e-12, atol=1e-12)
    if gated:
        q = cap["q"].reshape(n, SMALL.n_q, SMALL.head_dim)
        o = _sdpa_ref(q, cap["k"], cap["v"], True).reshape(n, -1)
        gate = torch.sigmoid(x @ t(W["w_attn_gate"]).T).numpy()
        assert np.allclose(cap["attn"], o * gate, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("gated", [False, True], ids=["plain", "gated"])
def test_input_embeddings_match_torch_rms_norm_concat(gated):
    _check_embed_layer(gated)


def test_zero_embedding_columns_reduce_to_the_plain_layer():
    # with the embedding half of Q/K/V zeroed, the tokens cannot matter and the
    # layer is the plain one over the hidden half
    hl, hm, hh = rand_states(8, SMALL.d, 44)
    W = _embed_model()
    d = SMALL.d
    for k in ("w_q", "w_k", "w_v"):
        W[k][:, :d] = 0.0
    plain = {k: (v[:, d:] if k in ("w_q", "w_k", "w_v") else v) for k, v in W.items()
             if k not in ("embed", "gamma_emb")}
    z1, h1, _ = OracleModel(SMALL, W).prefill_one(hl, hm, hh, tokens=np.arange(8) % VOCAB)
    z2, h2, _ = OracleModel(SMALL, W).prefill_one(hl, hm, hh, tokens=(np.arange(8) * 7 + 3) % VOCAB)
    z0, h0, _ = OracleModel(SMALL, plain).prefill_one(hl, hm, hh)
    assert np.allclose(h1, h0, rtol=1e-12, atol=1e-13) and np.allclose(h2, h0, rtol=1e-12, atol=1e-13)
    assert abs(z1 - z0) <= 1e-12 * max(1.0, abs(z0))


def test_embedding_rows_of_unused_tokens_do_not_matter():
    hl, hm, hh = rand_states(6, SMALL.d, 45)
    tok = np.array([1, 4, 4, 9, 1, 2])
    W = _embed_model()
    z1, h1, _ = OracleModel(SMALL, W).prefill_one(hl, hm, hh, tokens=tok)
    W2 = dict(W)
    W2["embed"] = W["embed"].copy()
    unused = np.setdiff1d(np.arange(VOCAB), tok)
    W2["embed"][unused] = 123.0
    z2, h2, _ = OracleModel(SMALL, W2).prefill_one(hl, hm, hh, tokens=tok)
    assert np.array_equal(h1, h2) and z1 == z2
    W2["embed"][4] += 1.0                      # a used row changes the result
    _, h3, _ = OracleModel(SMALL, W2).prefill_one(hl, hm, hh, tokens=tok)
    assert not np.allclose(h1, h3)


def test_input_embedding_steps_equal_prefill_recompute():
    n0, n1 = 5, 9
    hl, hm, hh = rand_states(n1, SMALL.d, 46)
    tok = np.random.default_rng(47).integers(0, VOCAB, n1)
    m = OracleModel(SMALL, _embed_model())
    _, _, st = m.prefill_one(hl[:n0], hm[:n0], hh[:n0], tokens=tok[:n0])
    for t in range(n0, n1):
        zs, hs = m.step_one(st, hl[t], hm[t], hh[t], token=int(tok[t]))
        zf, hf, _ = m.prefill_one(hl[:t + 1], hm[:t + 1], hh[:t + 1], tokens=tok[:t + 1])
        assert np.allclose(hs, hf[-1], rtol=1e-10, atol=1e-12)
        assert abs(zs - zf) <= 1e-10 * max(1.0, abs(zf))


# ------------------------------------------------------------- MLP probe

def _probe_weights(seed=21):
    r = np.random.default_rng(seed)
    d, h1 = SMALL.d, SMALL.head_hidden
    return {"probe_w1": r.standard_normal((h1, 2 * d)) * 0.3, "probe_b1": r.standard_normal(h1) * 0.3,
            "probe_w2": r.standard_normal(h1) * 0.3, "probe_b2": r.standard_normal(1) * 0.3}


def _torch_probe(W, h):
    t = torch.from_numpy
    mlp = torch.nn.Sequential(torch.nn.Linear(2 * SMALL.d, SMALL.head_hidden), torch.nn.ReLU(),
                              torch.nn.Linear(SMALL.head_hidden, 1)).double()
    with torch.no_grad():
        mlp[0].weight.copy_(t(W["probe_w1"])); mlp[0].bias.copy_(t(W["probe_b1"]))
        mlp[2].weight.copy_(t(W["probe_w2"])[None, :]); mlp[2].bias.copy_(t(W["probe_b2"]))
        x = torch.cat([t(h).mean(dim=0), t(h)[-1]])
        return float(mlp(x)[0])


def test_probe_matches_torch_mlp_on_mean_and_last():
    from oracle import OracleProbe
    W = _probe_weights()
    h = np.random.default_rng(22).standard_normal((11, SMALL.d)) * 2.0
    z, _ = OracleProbe(W).prefill_one(h)
    assert abs(z - _torch_probe(W, h)) <= 1e-12 * max(1.0, abs(z))


def test_probe_steps_equal_prefill_recompute():
    from oracle import OracleProbe
    W = _probe_weights()
    h = np.random.default_rng(23).standard_normal((9, SMALL.d))
    p = OracleProbe(W)
    _, st = p.prefill_one(h[:4])
    for t in range(4, 9):
        zs = p.step_one(st, h[t])
        zf, _ = OracleProbe(W).prefill_one(h[:t + 1])
        assert abs(zs - zf) <= 1e-12 * max(1.0, abs(zf))
        assert abs(zs - _torch_probe(W, h[:t + 1])) <= 1e-12 * max(1.0, abs(zs))


# ------------------------------------------------------------- draft model head

def test_draft_distribution_matches_torch_softmax():
    from oracle import draft_distribution
    r = np.random.default_rng(31)
    h = r.standard_normal((3, 16)) * 2.0
    w = r.standard_normal((50, 16))
    p = draft_distribution(h, w)
    ref = torch.softmax(torch.from_numpy(h) @ torch.from_numpy(w).T, dim=-1).numpy()
    assert np.allclose(p, ref, rtol=1e-12, atol=1e-15)
    assert np.allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-12)


# ------------------------------------------------------------- planted mistakes

def _fails(fn, *args):
    try:
        fn(*args)
    except AssertionError:
        return True
    return False


def _check_one_token(attn):
    r = np.random.default_rng(9)
    hq, hkv, hd = 8, 2, 4
    q, k, v = r.standard_normal((1, hq, hd)), r.standard_normal((1, hkv, hd)), r.standard_normal((1, hkv, hd))
    o = attn(q, k, v, np.array([0]), np.array([0]))
    for h in range(hq):
        assert np.array_equal(o[0, h], v[0, h // (hq // hkv)])


def test_planted_gqa_mapping_error_is_caught():
    def interleaved_groups(q, k, v, q_pos, k_pos, chunk=1024):
        idx = [h % k.shape[1] for h in range(q.shape[1])]
        group = q.shape[1] // k.shape[1]
        kk = np.stack([k[:, idx[h * group]] for h in range(k.shape[1])], axis=1)
        vv = np.stack([v[:, idx[h * group]] for h in range(k.shape[1])], axis=1)
        return causal_gqa_attention(q, kk, vv, q_pos, k_pos, chunk)
    assert _fails(_check_one_token, interleaved_groups)


def test_planted_rope_sign_error_is_caught():
    assert _fails(_check_rope_complex, lambda x, p, th: rope(x, -np.asarray(p), th))


def test_planted_rope_pairing_error_is_caught():
    def adjacent_pairs(x, positions, theta):
        hd = x.shape[-1]
        perm = np.concatenate([np.arange(0, hd, 2), np.arange(1, hd, 2)])
        inv = np.argsort(perm)
        return rope(x[..., perm], positions, theta)[..., inv]
    assert _fails(_check_rope_complex, adjacent_pairs)


def test_planted_missing_mask_is_caught():
    def unmasked(q, k, v, q_pos, k_pos, chunk=1024):
        return causal_gqa_attention(q, k, v, np.full_like(q_pos, 10 ** 9), k_pos, chunk)
    assert _fails(_check_sdpa, unmasked)


def test_planted_pool_order_error_is_caught():
    class SwappedPool(OracleModel):
        def prefill_one(self, h_low, h_mid, h_high):
            z, hd, st = super().prefill_one(h_low, h_mid, h_high)
            n = hd.shape[0]
            pooled = np.concatenate([hd[n - 1], hd.sum(axis=0) / n])[None, :]
            return float(self._head(pooled)[0]), hd, st
    assert _fails(_check_brute, SwappedPool, 5)


@pytest.mark.parametrize("mistake", ["no_sigmoid", "pre_norm_input", "one_minus"])
def test_planted_gate_mistakes_are_caught(monkeypatch, mistake):
    real = oracle_model.attention_output_gate

    def wrong(o, a, w):
        if mistake == "no_sigmoid":
            return o * (a @ w.T)
        if mistake == "pre_norm_input":      # gate from a rescaled input (norm skipped)
            return real(o, a * 1.7, w)
        return o * (1.0 - oracle_model.sigmoid(a @ w.T))
    monkeypatch.setattr(oracle_model, "attention_output_gate", wrong)
    assert _fails(_check_gated_layer)


@pytest.mark.parametrize("mistake", ["hidden_first", "no_norm", "no_gain"])
def test_planted_input_embedding_mistakes_are_caught(monkeypatch, mistake):
    real = oracle_model.embedded_attention_input

    def wrong(emb_rows, gamma_emb, a, eps):
        if mistake == "hidden_first":
            e, _ = real(emb_rows, gamma_emb, a, eps)
            return e, np.concatenate([a, e], axis=1)
        if mistake == "no_norm":
            return emb_rows * gamma_emb, np.concatenate([emb_rows * gamma_emb, a], axis=1)
        return real(emb_rows, np.ones_like(gamma_emb), a, eps)
    monkeypatch.setattr(oracle_model, "embedded_attention_input", wrong)
    assert _fails(_check_embed_layer)
