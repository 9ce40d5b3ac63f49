"""Seeded synthetic workloads for the OUTLETS draft-backbone + length-head path.

This module only draws random numbers and stores them in the storage formats
the path consumes (fp32, bf16 bit patterns, OCP e4m3 codes with bf16 row
scales).  It holds none of the method's arithmetic: no projection, norm,
attention, pooling or head.  Both the fp64 oracle and the GPU path take their
inputs from here and decode the stored formats independently.

Recipe (the same for every consumer):

* Every named tensor gets its own generator,
  ``numpy.random.default_rng(SeedSequence([seed, cfg_id, stream, index]))``.
* Linear weights are ``[out, in]`` row-major, drawn N(0, 0.02^2).  RMSNorm
  gains are 1 + 0.02 N(0, 1) (a gain drawn around zero would shrink every
  state and flip signs); head biases are N(0, 0.02^2).
* Target hidden states (the three depths h^(2), h^(N/2), h^(N-2) of
  Section 4.1) are N(0, 1) per element, multiplied by a per-depth scale
  (1, 4, 16 for the 8B/70B shapes; 1, 1, 1 for the tiny shape) to mimic the
  growth of the residual stream with depth.
* Prompt lengths are either uniform integers or
  ``clip(rint(exp(ln(median) + sigma * N(0, 1))), lo, hi)``.
* Draws are fp32 and rounded to the storage format with round-to-nearest-even.
  The e4m3 weights of the 70B shape use one bf16 scale per output row,
  ``s = bf16(max|W_row| / 448)``, and codes ``RNE(clamp(W / s, -448, 448))``.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

__all__ = [
    "DraftShape", "Workload", "WORKLOADS", "workload", "to_bf16_bits",
    "encode_e4m3", "make_weights", "make_lengths", "make_prompt_states",
    "make_step_states", "device_states", "WEIGHT_NAMES", "BIG_LINEARS", "GATE_NAME",
    "make_probe_weights", "make_lm_weights", "make_embed_weights", "make_prompt_tokens",
    "make_step_tokens",
]

# Linear layers of the draft backbone, the ones stored as e4m3 in the 70B
# shape.  Order is the order of their random streams.
BIG_LINEARS = ("w_proj", "w_q", "w_k", "w_v", "w_o", "w_gate", "w_up", "w_down")
WEIGHT_NAMES = BIG_LINEARS + (
    "gamma_attn", "gamma_mlp", "gamma_final", "head_w1", "head_b1",
    "head_w2", "head_b2")
# The attention output gate of Gated Attention (drawn only for workloads with
# ``attn_gate``; its stream follows the others so they do not change).
GATE_NAME = "w_attn_gate"


@dataclasses.dataclass(frozen=True)
class DraftShape:
    d: int            # draft hidden size (= target hidden size)
    n_q: int          # query heads
    n_kv: int         # key/value heads
    head_dim: int
    ffn: int          # SwiGLU inner width
    head_hidden: int  # width of the length head's hidden layer
    rope_theta: float
    rms_eps: float = 1e-5
    vocab: int = 0    # vocabulary of the draft model head (Eq. 2)

    def weight_shapes(self) -> Dict[str, Tuple[int, ...]]:
        d, hd = self.d, self.head_dim
        return {
            "w_proj": (d, 3 * d),
            "w_q": (self.n_q * hd, d),
            "w_k": (self.n_kv * hd, d),
            "w_v": (self.n_kv * hd, d),
            "w_o": (d, self.n_q * hd),
            "w_gate": (self.ffn, d),
            "w_up": (self.ffn, d),
            "w_down": (d, self.ffn),
            "w_attn_gate": (self.n_q * hd, d),
            "gamma_attn": (d,),
            "gamma_mlp": (d,),
            "gamma_final": (d,),
            "head_w1": (self.head_hidden, 2 * d),
            "head_b1": (self.head_hidden,),
            "head_w2": (self.head_hidden,),
            "head_b2": (1,),
        }


@dataclasses.dataclass(frozen=True)
class Workload:
    cfg_id: int
    name: str
    shape: DraftShape
    weight_fmt: str            # "f32" | "bf16" | "e4m3"
    act_fmt: str               # "f32" | "bf16"
    n_req: int
    lengths: Tuple             # ("uniform", lo, hi) | ("lognormal", median, sigma, lo, hi)
    input_scales: Tuple[float, float, float]
    steps: int = 0             # decode steps (re-prediction) after the prefill
    page_size: int = 16
    attn_gate: bool = False    # Gated Attention output gate in the draft layer
    input_embed: bool = False  # EAGLE-3 input embeddings: attention reads [emb ; f_ctx] (2d)

    @property
    def max_len(self) -> int:
        return int(self.lengths[-1])


SHAPE_TINY = DraftShape(d=256, n_q=4, n_kv=2, head_dim=64, ffn=688,
                        head_hidden=128, rope_theta=1e4, vocab=512)
# Llama-3 vocabulary (128,256 entries) for the draft model head of the 8B/70B shapes
SHAPE_8B = DraftShape(d=4096, n_q=32, n_kv=8, head_dim=128, ffn=14336,
                      head_hidden=1024, rope_theta=5e5, vocab=128256)
SHAPE_70B = DraftShape(d=8192, n_q=64, n_kv=8, head_dim=128, ffn=28672,
                       head_hidden=2048, rope_theta=5e5, vocab=128256)

WORKLOADS: Dict[int, Workload] = {
    0: Workload(0, "tiny-fp32", SHAPE_TINY, "f32", "f32", 4,
                ("uniform", 16, 64), (1.0, 1.0, 1.0), steps=8),
    1: Workload(1, "8b-bf16-prefill-b32", SHAPE_8B, "bf16", "bf16", 32,
                ("lognormal", 512, 1.0, 32, 4096), (1.0, 4.0, 16.0)),
    2: Workload(2, "8b-bf16-prefill-b256", SHAPE_8B, "bf16", "bf16", 256,
                ("lognormal", 1024, 1.2, 16, 8192), (1.0, 4.0, 16.0)),
    3: Workload(3, "8b-bf16-step-b512", SHAPE_8B, "bf16", "bf16", 512,
                ("uniform", 256, 8192), (1.0, 4.0, 16.0), steps=64),
    4: Workload(4, "70b-e4m3-prefill-b64", SHAPE_70B, "e4m3", "bf16", 64,
                ("lognormal", 2048, 1.0, 64, 16384), (1.0, 4.0, 16.0)),
}


def workload(cfg_id: int, **overrides) -> Workload:
    """The named workload, optionally with fields replaced (e.g. a smaller
    request count or a reduced shape for parity tests)."""
    w = WORKLOADS[cfg_id]
    return dataclasses.replace(w, **overrides) if overrides else w


# ---------------------------------------------------------------- encodings

def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 values -> bf16 bit patterns (uint16), round to nearest even.
    Inputs are finite by construction."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def _bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def encode_e4m3(w: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Per-output-row OCP e4m3 encoding of an fp32 ``[out, in]`` matrix.

    Returns ``(codes uint8 [out, in], scale_bits uint16 [out])``.  The scale
    is the bf16 rounding of ``max|row| / 448``; codes are the round-to-nearest
    -even e4m3 values of ``row / scale`` clamped to the finite range."""
    import torch  # the encoder uses torch's float8_e4m3fn conversion (RNE)
    w = np.ascontiguousarray(w, dtype=np.float32)
    amax = np.abs(w).max(axis=1)
    amax = np.where(amax > 0, amax, np.float32(1.0))
    s_bits = to_bf16_bits(amax / np.float32(448.0))
    s = _bf16_bits_to_f32(s_bits)
    q = np.clip(w / s[:, None], -448.0, 448.0).astype(np.float32)
    codes = torch.from_numpy(q).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return codes.copy(), s_bits


# ---------------------------------------------------------------- draws

def _rng(seed: int, cfg_id: int, stream: int, index: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, cfg_id, stream, index]))


def make_weights(wl: Workload, seed: int = 0) -> Dict[str, object]:
    """All weights of the draft layer and the length head, in storage format.

    Returns a dict ``name -> array``.  For ``f32`` arrays are float32; for
    ``bf16`` they are uint16 bit patterns; for ``e4m3`` the eight big linears
    are ``(codes uint8, scale_bits uint16)`` tuples and the rest bf16 bits.
    ``out['_fmt']`` records the format of each entry."""
    shapes = wl.shape.weight_shapes()
    if wl.input_embed:
        # the attention projections read [normed embedding ; normed f_ctx]
        for name in ("w_q", "w_k", "w_v", GATE_NAME):
            shapes[name] = (shapes[name][0], 2 * wl.shape.d)
    out: Dict[str, object] = {}
    fmt: Dict[str, str] = {}
    names = list(enumerate(WEIGHT_NAMES))
    if wl.attn_gate:
        names.append((len(WEIGHT_NAMES), GATE_NAME))
    for stream, name in names:
        rng = _rng(seed, wl.cfg_id, stream)
        shp = shapes[name]
        x = rng.standard_normal(shp, dtype=np.float32)
        if name.startswith("gamma"):
            x = np.float32(1.0) + np.float32(0.02) * x
        else:
            x = np.float32(0.02) * x
        if wl.weight_fmt == "f32":
            out[name], fmt[name] = x, "f32"
        elif wl.weight_fmt == "e4m3" and (name in BIG_LINEARS or name == GATE_NAME):
            out[name], fmt[name] = encode_e4m3(x), "e4m3"
        else:
            out[name], fmt[name] = to_bf16_bits(x), "bf16"
        del x
    if wl.input_embed:
        emb = make_embed_weights(wl, seed)
        fmt.update(emb.pop("_fmt"))
        out.update(emb)
    out["_fmt"] = fmt
    return out


def make_probe_weights(wl: Workload, seed: int = 0) -> Dict[str, object]:
    """Weights of the MLP-probe baseline (same form as the length head:
    probe_w1 [H1, 2d], probe_b1 [H1], probe_w2 [H1], probe_b2 [1]), drawn
    N(0, 0.02^2) from streams after every other weight's, stored in the
    small-weight format.  Returns a dict with its own ``_fmt`` entries."""
    d, h1 = wl.shape.d, wl.shape.head_hidden
    shapes = {"probe_w1": (h1, 2 * d), "probe_b1": (h1,), "probe_w2": (h1,), "probe_b2": (1,)}
    out: Dict[str, object] = {}
    fmt: Dict[str, str] = {}
    for k, (name, shp) in enumerate(shapes.items()):
        rng = _rng(seed, wl.cfg_id, len(WEIGHT_NAMES) + 1 + k)
        x = np.float32(0.02) * rng.standard_normal(shp, dtype=np.float32)
        if wl.weight_fmt == "f32":
            out[name], fmt[name] = x, "f32"
        else:
            out[name], fmt[name] = to_bf16_bits(x), "bf16"
    out["_fmt"] = fmt
    return out


def make_lm_weights(wl: Workload, seed: int = 0) -> Dict[str, object]:
    """W_lm [vocab, d] of the draft model head (Eq. 2), N(0, 0.02^2), from the
    stream after the probe's, stored like the big linears (``w_lm``; for
    e4m3 a ``(codes, scale_bits)`` tuple).  Returns a dict with ``_fmt``."""
    v, d = wl.shape.vocab, wl.shape.d
    rng = _rng(seed, wl.cfg_id, len(WEIGHT_NAMES) + 5)
    x = np.float32(0.02) * rng.standard_normal((v, d), dtype=np.float32)
    if wl.weight_fmt == "f32":
        return {"w_lm": x, "_fmt": {"w_lm": "f32"}}
    if wl.weight_fmt == "e4m3":
        return {"w_lm": encode_e4m3(x), "_fmt": {"w_lm": "e4m3"}}
    return {"w_lm": to_bf16_bits(x), "_fmt": {"w_lm": "bf16"}}


def make_embed_weights(wl: Workload, seed: int = 0) -> Dict[str, object]:
    """The target model's (frozen) token embedding table ``embed`` [vocab, d]
    (N(0, 0.02^2), activation format) and the draft layer's RMSNorm gain for
    it, ``gamma_emb`` [d] (1 + 0.02 N(0, 1), small-weight format), for the
    EAGLE-3 input-embedding concat.  Streams follow the draft head's."""
    v, d = wl.shape.vocab, wl.shape.d
    e = np.float32(0.02) * _rng(seed, wl.cfg_id, len(WEIGHT_NAMES) + 6).standard_normal((v, d), dtype=np.float32)
    g = np.float32(1.0) + np.float32(0.02) * _rng(seed, wl.cfg_id, len(WEIGHT_NAMES) + 7).standard_normal(d, dtype=np.float32)
    if wl.act_fmt == "f32":
        return {"embed": e, "gamma_emb": g, "_fmt": {"embed": "f32", "gamma_emb": "f32"}}
    return {"embed": to_bf16_bits(e), "gamma_emb": to_bf16_bits(g), "_fmt": {"embed": "bf16", "gamma_emb": "bf16"}}


def make_prompt_tokens(wl: Workload, lengths, seed: int = 0,
                       requests: Optional[List[int]] = None) -> np.ndarray:
    """Prompt token ids (int32, uniform over the vocabulary), packed like
    make_prompt_states; request ``i`` draws from its own generator."""
    lengths = np.asarray(lengths)
    idx = range(len(lengths)) if requests is None else requests
    parts = [_rng(seed, wl.cfg_id, 500, int(i)).integers(0, wl.shape.vocab, int(lengths[i]))
             for i in idx]
    return (np.concatenate(parts) if parts else np.zeros(0)).astype(np.int32)


def make_step_tokens(wl: Workload, n_req: int, step: int, seed: int = 0,
                     requests: Optional[List[int]] = None) -> np.ndarray:
    """Token ids generated at decode step ``step``, one per request."""
    idx = range(n_req) if requests is None else requests
    return np.array([_rng(seed, wl.cfg_id, 501, step * 1_000_003 + int(i)).integers(0, wl.shape.vocab)
                     for i in idx], dtype=np.int32)


def make_lengths(wl: Workload, seed: int = 0, n_req: Optional[int] = None) -> np.ndarray:
    """Prompt lengths (int32 [n_req]) per the workload's length law."""
    n = wl.n_req if n_req is None else n_req
    rng = _rng(seed, wl.cfg_id, 50)
    law = wl.lengths
    if law[0] == "uniform":
        lo, hi = int(law[1]), int(law[2])
        v = rng.integers(lo, hi + 1, size=n)
    elif law[0] == "lognormal":
        med, sigma, lo, hi = float(law[1]), float(law[2]), int(law[3]), int(law[4])
        z = rng.standard_normal(n)
        v = np.clip(np.rint(np.exp(np.log(med) + sigma * z)), lo, hi)
    else:
        raise ValueError(f"unknown length law {law[0]!r}")
    return v.astype(np.int32)


def _states(rng: np.random.Generator, rows: int, d: int, scale: float, fmt: str) -> np.ndarray:
    x = rng.standard_normal((rows, d), dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return x if fmt == "f32" else to_bf16_bits(x)


def make_prompt_states(wl: Workload, lengths, seed: int = 0,
                       requests: Optional[List[int]] = None) -> List[np.ndarray]:
    """Target hidden states (low, mid, high) for the prompts, packed in
    request order: three arrays ``[sum(lengths), d]``.

    Request ``i`` always draws from its own generator, so any subset of the
    requests (``requests=[...]`` indexes into ``lengths``) reproduces exactly
    the rows the full batch holds for them."""
    lengths = np.asarray(lengths)
    idx = range(len(lengths)) if requests is None else requests
    d = wl.shape.d
    out = []
    for depth in range(3):
        parts = [_states(_rng(seed, wl.cfg_id, 100 + depth, int(i)), int(lengths[i]), d,
                         wl.input_scales[depth], wl.act_fmt) for i in idx]
        out.append(np.concatenate(parts, axis=0) if parts else
                   np.zeros((0, d), np.float32 if wl.act_fmt == "f32" else np.uint16))
    return out


def make_step_states(wl: Workload, n_req: int, step: int, seed: int = 0,
                     requests: Optional[List[int]] = None) -> List[np.ndarray]:
    """States of the token generated at decode step ``step`` (1-based), one
    row per request: three arrays ``[n_req or len(requests), d]``.  Row ``i``
    of the full batch is drawn by its own generator, so subsets reproduce it."""
    idx = range(n_req) if requests is None else requests
    d = wl.shape.d
    out = []
    for depth in range(3):
        rows = [_states(_rng(seed, wl.cfg_id, 200 + depth, step * 1_000_003 + int(i)), 1, d,
                        wl.input_scales[depth], wl.act_fmt) for i in idx]
        out.append(np.concatenate(rows, axis=0) if rows else
                   np.zeros((0, d), np.float32 if wl.act_fmt == "f32" else np.uint16))
    return out


def device_states(wl: Workload, rows: int, seed: int, stream: int, index: int, device="cuda"):
    """Target states drawn directly on the GPU (torch's seeded normal
    generator), for benchmark workloads too large to draw on the host in
    reasonable time: three tensors [rows, d] in the workload's activation
    format, N(0, 1) times the per-depth scales.  The values differ from
    make_prompt_states' (another generator); parity tests use the host draws."""
    import torch
    g = torch.Generator(device=device)
    out = []
    for depth in range(3):
        g.manual_seed(int(np.random.SeedSequence([seed, wl.cfg_id, stream + depth, index]).generate_state(1)[0]))
        x = torch.randn((rows, wl.shape.d), generator=g, device=device, dtype=torch.float32)
        x *= wl.input_scales[depth]
        out.append(x if wl.act_fmt == "f32" else x.to(torch.bfloat16))
    return out
