"""fp64 CPU oracle of the OUTLETS draft backbone and length head.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this module.  It shares no
code with the HIP library and imports nothing from it.

Everything is float64, one request at a time, in the order the paper
describes (Section 4.1 backbone, Section 4.2 heads, Section 3.2 static and
dynamic prediction).  Where the paper leaves a detail open the reading used
here is stated next to the code:

* Fusion (Eq. 1): f_ctx = W_proj Concat(h_low, h_mid, h_high), no bias, the
  concatenation in low, mid, high order.
* Draft decoder layer (Section 4.1): a Llama-style pre-norm layer.  The
  residual stream starts at f_ctx; RMSNorm (eps 1e-5) before attention and
  before the SwiGLU MLP; bias-free linears; rotate-half RoPE with frequencies
  theta^(-2c/hd) and no frequency rescaling; grouped-query attention where
  query head h reads key/value head floor(h / (n_q / n_kv)); causal within
  a request.
* Gated Attention (Section 4.1 names it and cites its source without giving
  a formula): optional, off unless the weights carry ``w_attn_gate``.  The
  reading taken is the elementwise output gate of the cited work: each
  attention output element, per query head and channel, is multiplied by
  sigmoid of a bias-free linear map of the same normed input that feeds
  Q/K/V, before the heads are concatenated into W_o.
* Input embeddings (the EAGLE-3 component the Section 5 ablation lists,
  no formula given): optional, off unless the weights carry ``embed``.  The
  reading taken is EAGLE-3's: the attention block reads the 2d-wide row
  [RMSNorm(embed[token]) * gamma_emb ; RMSNorm(f_ctx) * gamma_attn], so
  W_q, W_k, W_v (and the gate) have 2d input columns, embedding columns
  first; the residual stream still starts at f_ctx.  Which token is paired
  with a row is the caller's choice (EAGLE-3 pairs a position with the
  token that follows it).
* h^draft is the final RMSNorm of the layer output (both heads read it).
* Length head (Section 4.2): the pooled state p = [mean over the request's
  tokens of h^draft ; h^draft of the newest token] goes through
  Linear(2d, H1) + ReLU + Linear(H1, 1), both with biases; the output z_hat
  estimates log(1 + remaining length) (natural log).
* Dynamic prediction (Section 3.2): a decode step appends one token at
  position n + t - 1, attends over every cached key plus itself, updates the
  running mean over all tokens so far (prompt and generated), and re-runs the
  head.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .formats import decode_states, decode_weight

WEIGHT_KEYS = ("w_proj", "w_q", "w_k", "w_v", "w_o", "w_gate", "w_up", "w_down",
               "gamma_attn", "gamma_mlp", "gamma_final", "head_w1", "head_b1",
               "head_w2", "head_b2")


@dataclasses.dataclass(frozen=True)
class OracleShape:
    d: int
    n_q: int
    n_kv: int
    head_dim: int
    ffn: int
    head_hidden: int
    rope_theta: float
    rms_eps: float = 1e-5


def decode_weights(stored: Dict[str, object]) -> Dict[str, np.ndarray]:
    """Stored weights (as the seeded generator returns them) -> float64.
    The attention output gate ``w_attn_gate`` and the input-embedding table
    ``embed`` with its gain ``gamma_emb`` are carried over when present."""
    fmt = stored["_fmt"]
    keys = WEIGHT_KEYS + tuple(k for k in ("w_attn_gate", "embed", "gamma_emb") if k in stored)
    return {k: decode_weight(stored[k], fmt[k]) for k in keys}


# ------------------------------------------------------------------ layers

def fuse(w_proj: np.ndarray, h_low: np.ndarray, h_mid: np.ndarray,
         h_high: np.ndarray) -> np.ndarray:
    """Eq. 1: f_ctx = W_proj . Concat(h_low, h_mid, h_high); rows are tokens."""
    x = np.concatenate([h_low, h_mid, h_high], axis=1)
    return x @ w_proj.T


def rms_norm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * gamma."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gamma


def rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of x [n, heads, hd] at integer positions.

    Channel pair (c, c + hd/2) is rotated by the angle p * theta^(-2c/hd)."""
    hd = x.shape[-1]
    half = hd // 2
    c = np.arange(half, dtype=np.float64)
    omega = theta ** (-2.0 * c / hd)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * omega[None, :]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def causal_gqa_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                         q_pos: np.ndarray, k_pos: np.ndarray,
                         chunk: int = 1024) -> np.ndarray:
    """softmax(q k^T / sqrt(hd)) v per query head, keys with position > the
    query's position masked out.  q [nq_tok, Hq, hd]; k, v [nk_tok, Hkv, hd].

    Query rows are independent, so they are processed ``chunk`` at a time only
    to bound memory.  Keys later than every query of a chunk are masked for
    all of its rows (weight exactly zero), so they are left out of that
    chunk's scores."""
    n_tok, n_q, hd = q.shape
    n_kv = k.shape[1]
    group = n_q // n_kv
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(hd)
    for s in range(0, n_tok, chunk):
        e = min(n_tok, s + chunk)
        qp = q_pos[s:e]
        keep = k_pos <= qp.max()
        kp, kc, vc = (k_pos, k, v) if keep.all() else (k_pos[keep], k[keep], v[keep])
        masked = kp[None, :] > qp[:, None]
        for h in range(n_q):
            g = h // group
            scores = q[s:e, h, :] @ kc[:, g, :].T
            scores *= scale
            np.putmask(scores, masked, -np.inf)
            scores -= scores.max(axis=1, keepdims=True)
            np.exp(scores, out=scores)
            scores /= scores.sum(axis=1, keepdims=True)
            out[s:e, h, :] = scores @ vc[:, g, :]
    return out


def silu(u: np.ndarray) -> np.ndarray:
    return u / (1.0 + np.exp(-u))


def sigmoid(u: np.ndarray) -> np.ndarray:
    return 1.0 / (1.0 + np.exp(-u))


def attention_output_gate(o: np.ndarray, a: np.ndarray, w_attn_gate: np.ndarray) -> np.ndarray:
    """Gated Attention output gate: o [n, n_q*hd] (heads concatenated) times
    sigmoid(a W_g^T) elementwise, a the normed layer input [n, d]."""
    return o * sigmoid(a @ w_attn_gate.T)


def embedded_attention_input(emb_rows: np.ndarray, gamma_emb: np.ndarray, a: np.ndarray,
                             eps: float) -> Tuple[np.ndarray, np.ndarray]:
    """EAGLE-3 input embeddings: e = RMSNorm(emb_rows) * gamma_emb and the
    attention block's input row [e ; a], a the normed f_ctx.  Returns (e, x)."""
    e = rms_norm(emb_rows, gamma_emb, eps)
    return e, np.concatenate([e, a], axis=1)


def swiglu_mlp(b: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray,
               w_down: np.ndarray) -> np.ndarray:
    """(silu(b W_gate^T) * (b W_up^T)) W_down^T."""
    return (silu(b @ w_gate.T) * (b @ w_up.T)) @ w_down.T


def length_head(p: np.ndarray, w1: np.ndarray, b1: np.ndarray, w2: np.ndarray,
                b2: np.ndarray) -> np.ndarray:
    """MLP_len of Section 4.2: z_hat = w2 . relu(W1 p + b1) + b2, rows of p."""
    u = np.maximum(p @ w1.T + b1, 0.0)
    return u @ w2 + b2[0]


def draft_distribution(h_draft: np.ndarray, w_lm: np.ndarray) -> np.ndarray:
    """Eq. 2, the draft model head: P_draft(y_{t+1} | y_{1:t}) =
    softmax(W_lm h_t^draft) over the vocabulary, rows of h_draft."""
    logits = h_draft @ w_lm.T
    e = np.exp(logits - logits.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


# ------------------------------------------------------------------ model

@dataclasses.dataclass
class RequestState:
    """Per-request draft KV cache and running pool, as dynamic prediction needs."""
    k: np.ndarray          # [n, Hkv, hd], keys after RoPE
    v: np.ndarray          # [n, Hkv, hd]
    pool_sum: np.ndarray   # [d], sum of h^draft over every token so far
    count: int             # tokens so far (prompt + generated)


class OracleModel:
    def __init__(self, shape: OracleShape, weights: Dict[str, np.ndarray]):
        self.s = shape
        self.w = weights

    # one pass of the draft layer over new tokens at known positions
    def _layer(self, h_low, h_mid, h_high, positions, k_prev, v_prev, k_pos_prev, capture=None,
               tokens=None):
        s, w = self.s, self.w
        n = h_low.shape[0]
        f = fuse(w["w_proj"], h_low, h_mid, h_high)
        a = rms_norm(f, w["gamma_attn"], s.rms_eps)
        if "embed" in w:
            e, x_attn = embedded_attention_input(w["embed"][np.asarray(tokens)], w["gamma_emb"], a,
                                                 s.rms_eps)
        else:
            e, x_attn = None, a
        q = (x_attn @ w["w_q"].T).reshape(n, s.n_q, s.head_dim)
        k = (x_attn @ w["w_k"].T).reshape(n, s.n_kv, s.head_dim)
        v = (x_attn @ w["w_v"].T).reshape(n, s.n_kv, s.head_dim)
        q = rope(q, positions, s.rope_theta)
        k = rope(k, positions, s.rope_theta)
        k_all = np.concatenate([k_prev, k], axis=0)
        v_all = np.concatenate([v_prev, v], axis=0)
        k_pos = np.concatenate([k_pos_prev, positions])
        o = causal_gqa_attention(q, k_all, v_all, positions, k_pos).reshape(n, s.n_q * s.head_dim)
        if "w_attn_gate" in w:
            o = attention_output_gate(o, x_attn, w["w_attn_gate"])
        x1 = f + o @ w["w_o"].T
        b = rms_norm(x1, w["gamma_mlp"], s.rms_eps)
        x2 = x1 + swiglu_mlp(b, w["w_gate"], w["w_up"], w["w_down"])
        h_draft = rms_norm(x2, w["gamma_final"], s.rms_eps)
        if capture is not None:
            # capture["_only"] (a set of names) limits what is stored; the
            # SwiGLU product is recomputed only when it is asked for
            only = capture.get("_only")
            want = lambda name: only is None or name in only  # noqa: E731
            vals = dict(fused=f, norm_attn=a, q=q.reshape(n, -1), k=k, v=v, attn=o, x1=x1,
                        norm_mlp=b, x2=x2, hdraft=h_draft)
            if e is not None:
                vals["norm_emb"] = e
            capture.update({k_: v_ for k_, v_ in vals.items() if want(k_)})
            if want("mlp_act"):
                capture["mlp_act"] = silu(b @ w["w_gate"].T) * (b @ w["w_up"].T)
        return h_draft, k_all, v_all

    def _head(self, pooled: np.ndarray) -> np.ndarray:
        w = self.w
        return length_head(pooled, w["head_w1"], w["head_b1"], w["head_w2"], w["head_b2"])

    def prefill_one(self, h_low, h_mid, h_high, capture=None, tokens=None
                    ) -> Tuple[float, np.ndarray, RequestState]:
        """Static prediction (Section 3.2, t = 0) for one prompt of n tokens.
        ``capture`` (a dict) receives the layer's intermediate activations;
        ``tokens`` [n] are the ids paired with the rows (input embeddings)."""
        s = self.s
        n = h_low.shape[0]
        empty = np.zeros((0, s.n_kv, s.head_dim))
        pos = np.arange(n)
        h_draft, k, v = self._layer(h_low, h_mid, h_high, pos, empty, empty,
                                    np.zeros(0, dtype=np.int64), capture, tokens)
        pool_sum = h_draft.sum(axis=0)
        pooled = np.concatenate([pool_sum / n, h_draft[n - 1]])[None, :]
        if capture is not None:
            capture["pooled"] = pooled[0]
        z = float(self._head(pooled)[0])
        return z, h_draft, RequestState(k, v, pool_sum, n)

    def step_one(self, st: RequestState, h_low, h_mid, h_high, token=None, capture=None
                 ) -> Tuple[float, np.ndarray]:
        """Dynamic prediction (Section 3.2, t >= 1): one new token for one request.
        Updates ``st`` in place.  ``capture`` (a dict) receives the layer's
        intermediate activations of the new token, as in ``prefill_one``."""
        p = st.count
        pos = np.array([p])
        h_draft, k, v = self._layer(h_low[None, :], h_mid[None, :], h_high[None, :], pos,
                                    st.k, st.v, np.arange(p), capture,
                                    None if token is None else [token])
        st.k, st.v = k, v
        st.pool_sum = st.pool_sum + h_draft[0]
        st.count = p + 1
        pooled = np.concatenate([st.pool_sum / st.count, h_draft[0]])[None, :]
        if capture is not None:
            capture["pooled"] = pooled[0]
        return float(self._head(pooled)[0]), h_draft[0]

    # batched API: requests one by one, packed outputs
    def prefill(self, lens: Sequence[int], h_low, h_mid, h_high, tokens=None):
        """Packed prompts -> (z [B], h_draft [T, d], states)."""
        offs = np.concatenate([[0], np.cumsum(np.asarray(lens, dtype=np.int64))])
        zs, hs, states = [], [], []
        for i in range(len(lens)):
            a, b = offs[i], offs[i + 1]
            z, h, st = self.prefill_one(h_low[a:b], h_mid[a:b], h_high[a:b],
                                        tokens=None if tokens is None else tokens[a:b])
            zs.append(z)
            hs.append(h)
            states.append(st)
        hd = np.concatenate(hs, axis=0) if hs else np.zeros((0, self.s.d))
        return np.array(zs), hd, states

    def step(self, states: List[RequestState], h_low, h_mid, h_high, tokens=None, captures=None):
        """One decode step for every request in ``states`` (rows in order);
        ``captures`` (a list of dicts, one per request) receive the
        intermediates."""
        zs, hs = [], []
        for i, st in enumerate(states):
            z, h = self.step_one(st, h_low[i], h_mid[i], h_high[i],
                                 None if tokens is None else int(tokens[i]),
                                 None if captures is None else captures[i])
            zs.append(z)
            hs.append(h)
        return np.array(zs), (np.stack(hs) if hs else np.zeros((0, self.s.d)))


# ------------------------------------------------------------------ MLP probe

PROBE_KEYS = ("probe_w1", "probe_b1", "probe_w2", "probe_b2")


@dataclasses.dataclass
class ProbeState:
    pool_sum: np.ndarray
    count: int


class OracleProbe:
    """The MLP-probe baseline of Section 5.1 (an MLP regressor on the frozen
    target model's hidden states, no draft layer).  Reading: the probe sees
    one target-state tensor and uses the length head's input and form,
    [mean over the tokens so far ; newest token] -> Linear + ReLU -> Linear."""

    def __init__(self, weights: Dict[str, np.ndarray]):
        self.w = weights

    def _z(self, pooled: np.ndarray) -> float:
        w = self.w
        return float(length_head(pooled[None, :], w["probe_w1"], w["probe_b1"], w["probe_w2"],
                                 w["probe_b2"])[0])

    def prefill_one(self, h: np.ndarray) -> Tuple[float, ProbeState]:
        n = h.shape[0]
        s = h.sum(axis=0)
        return self._z(np.concatenate([s / n, h[n - 1]])), ProbeState(s, n)

    def step_one(self, st: ProbeState, h_row: np.ndarray) -> float:
        st.pool_sum = st.pool_sum + h_row
        st.count += 1
        return self._z(np.concatenate([st.pool_sum / st.count, h_row]))


def probe_from_stored(stored: Dict[str, object]) -> OracleProbe:
    fmt = stored["_fmt"]
    return OracleProbe({k: decode_weight(stored[k], fmt[k]) for k in PROBE_KEYS})


def oracle_from_workload(wl, stored_weights) -> OracleModel:
    """Build the oracle for a workload description (duck-typed: ``wl.shape``)."""
    sh = wl.shape
    shape = OracleShape(sh.d, sh.n_q, sh.n_kv, sh.head_dim, sh.ffn, sh.head_hidden,
                        sh.rope_theta, sh.rms_eps)
    return OracleModel(shape, decode_weights(stored_weights))


def states_to_f64(arrs, act_fmt: str):
    return [decode_states(a, act_fmt) for a in arrs]
