"""Torch-facing wrapper of the C ABI: owns the device copies of the weights
and calls outlets_predict_prefill / outlets_predict_step on torch tensors.

PyTorch is used for device memory and streams only; every step of the path
runs in ``liboutlets.so``.
"""
from __future__ import annotations

import ctypes as C
from typing import Dict, Optional, Sequence

import numpy as np
import torch

from . import binding as B

_FMT = {"f32": B.OUTLETS_FMT_F32, "bf16": B.OUTLETS_FMT_BF16, "e4m3": B.OUTLETS_FMT_E4M3}
BIG_LINEARS = ("w_proj", "w_q", "w_k", "w_v", "w_o", "w_gate", "w_up", "w_down")
SMALL = ("gamma_attn", "gamma_mlp", "gamma_final", "head_w1", "head_b1", "head_w2", "head_b2")
GATE_NAME = "w_attn_gate"    # optional Gated Attention output-gate projection
PROBE = ("probe_w1", "probe_b1", "probe_w2", "probe_b2")   # optional MLP-probe baseline
EMBED = ("embed", "gamma_emb")   # optional EAGLE-3 input embeddings


def to_device(arr, device="cuda") -> torch.Tensor:
    """Stored array -> device tensor: float32 stays float32, uint16 holds bf16
    bit patterns, uint8 holds e4m3 codes (kept as raw bytes)."""
    a = np.ascontiguousarray(arr)
    if a.dtype == np.float32:
        t = torch.from_numpy(a)
    elif a.dtype == np.uint16:
        t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    elif a.dtype == np.uint8:
        t = torch.from_numpy(a)
    else:
        raise TypeError(f"unsupported stored dtype {a.dtype}")
    return t.to(device)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _tokens_ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if t.dtype != torch.int32 or not t.is_cuda or not t.is_contiguous():
        raise TypeError("token ids must be a contiguous int32 device tensor")
    return t.data_ptr()


def _stream_ptr(stream: Optional[torch.cuda.Stream]) -> Optional[int]:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream or None


class OutletsPredictor:
    def __init__(self, shape, weight_fmt: str, act_fmt: str, weights: Dict[str, object], *,
                 max_slots: int, max_seq_len: int, num_pages: int, max_batch_tokens: int,
                 max_batch_requests: int, keep_intermediates: bool = False, device: int = 0):
        B.lib()
        self.shape = shape
        self.weight_fmt, self.act_fmt = weight_fmt, act_fmt
        self.device = torch.device("cuda", device)
        self.act_dtype = torch.float32 if act_fmt == "f32" else torch.bfloat16
        self.tensors = {}
        w = B.outlets_weights()
        for name in BIG_LINEARS:
            entry = weights[name]
            if weight_fmt == "e4m3":
                codes, scale = entry
                self.tensors[name] = to_device(codes, self.device)
                self.tensors["s" + name[1:]] = to_device(scale, self.device)
                setattr(w, "s" + name[1:], _ptr(self.tensors["s" + name[1:]]))
            else:
                self.tensors[name] = to_device(entry, self.device)
            setattr(w, name, _ptr(self.tensors[name]))
        for name in SMALL:
            self.tensors[name] = to_device(weights[name], self.device)
            setattr(w, name, _ptr(self.tensors[name]))
        if weights.get(GATE_NAME) is not None:      # Gated Attention output gate
            entry = weights[GATE_NAME]
            if weight_fmt == "e4m3":
                codes, scale = entry
                self.tensors[GATE_NAME] = to_device(codes, self.device)
                self.tensors["s_attn_gate"] = to_device(scale, self.device)
                w.s_attn_gate = _ptr(self.tensors["s_attn_gate"])
            else:
                self.tensors[GATE_NAME] = to_device(entry, self.device)
            w.w_attn_gate = _ptr(self.tensors[GATE_NAME])
        self.vocab = 0
        if weights.get("w_lm") is not None:              # draft model head (Eq. 2)
            entry = weights["w_lm"]
            if weight_fmt == "e4m3":
                codes, scale = entry
                self.tensors["w_lm"] = to_device(codes, self.device)
                self.tensors["s_lm"] = to_device(scale, self.device)
                w.s_lm = _ptr(self.tensors["s_lm"])
            else:
                self.tensors["w_lm"] = to_device(entry, self.device)
            w.w_lm = _ptr(self.tensors["w_lm"])
            self.vocab = int(shape.vocab)
        self.input_embed = weights.get("embed") is not None
        for name in EMBED:                               # EAGLE-3 input embeddings
            if weights.get(name) is not None:            # (the library checks both are given)
                self.tensors[name] = to_device(weights[name], self.device)
                setattr(w, name, _ptr(self.tensors[name]))
        if self.input_embed:
            self.vocab = int(shape.vocab)
        if weights.get("probe_w1") is not None:          # MLP-probe baseline
            for name in PROBE:
                self.tensors[name] = to_device(weights[name], self.device)
                setattr(w, name, _ptr(self.tensors[name]))
        self._w = w
        cfg = B.outlets_config()
        cfg.d_model, cfg.n_q_heads, cfg.n_kv_heads = shape.d, shape.n_q, shape.n_kv
        cfg.head_dim, cfg.ffn_dim, cfg.head_hidden = shape.head_dim, shape.ffn, shape.head_hidden
        cfg.rope_theta, cfg.rms_eps = shape.rope_theta, shape.rms_eps
        cfg.weight_fmt, cfg.act_fmt, cfg.page_size = _FMT[weight_fmt], _FMT[act_fmt], 16
        cfg.max_slots, cfg.max_seq_len, cfg.num_pages = max_slots, max_seq_len, num_pages
        cfg.max_batch_tokens, cfg.max_batch_requests = max_batch_tokens, max_batch_requests
        cfg.keep_intermediates = int(bool(keep_intermediates))
        cfg.vocab = self.vocab
        self.cfg = cfg
        torch.cuda.synchronize(self.device)
        self.ctx = B.outlets_create(cfg, w, device)

    # ------------------------------------------------------------ calls
    def prefill(self, slots: Sequence[int], lens: Sequence[int], h_low: torch.Tensor,
                h_mid: torch.Tensor, h_high: torch.Tensor, row_stride: Optional[int] = None,
                want_hdraft: bool = False, z_out: Optional[torch.Tensor] = None,
                hdraft_out: Optional[torch.Tensor] = None, stream=None,
                tokens: Optional[torch.Tensor] = None):
        """``tokens``: device int32 [T] ids paired with the rows (input embeddings)."""
        n, T = len(slots), int(sum(int(x) for x in lens))
        if z_out is None:
            z_out = torch.empty(max(n, 1), dtype=torch.float32, device=self.device)
        if want_hdraft and hdraft_out is None:
            hdraft_out = torch.empty((max(T, 1), self.shape.d), dtype=self.act_dtype, device=self.device)
        stride = h_low.stride(0) if row_stride is None else row_stride
        rc = B.outlets_predict_prefill(self.ctx, list(slots), list(lens), h_low.data_ptr(), h_mid.data_ptr(),
                                       h_high.data_ptr(), stride, _tokens_ptr(tokens), z_out.data_ptr(),
                                       _ptr(hdraft_out), _stream_ptr(stream))
        B.check(rc, "outlets_predict_prefill")
        return z_out[:n], (hdraft_out[:T] if hdraft_out is not None else None)

    def step(self, slots: Sequence[int], h_low: torch.Tensor, h_mid: torch.Tensor,
             h_high: torch.Tensor, row_stride: Optional[int] = None, want_hdraft: bool = False,
             z_out: Optional[torch.Tensor] = None, hdraft_out: Optional[torch.Tensor] = None,
             stream=None, tokens: Optional[torch.Tensor] = None, noalloc: bool = False):
        """``noalloc``: run outlets_predict_step_noalloc (per-call buffers in
        the library's static scratch; pass z_out / hdraft_out to keep the
        call itself free of allocations)."""
        n = len(slots)
        if z_out is None:
            z_out = torch.empty(max(n, 1), dtype=torch.float32, device=self.device)
        if want_hdraft and hdraft_out is None:
            hdraft_out = torch.empty((max(n, 1), self.shape.d), dtype=self.act_dtype, device=self.device)
        stride = h_low.stride(0) if row_stride is None else row_stride
        fn = B.outlets_predict_step_noalloc if noalloc else B.outlets_predict_step
        rc = fn(self.ctx, list(slots), h_low.data_ptr(), h_mid.data_ptr(), h_high.data_ptr(), stride,
                _tokens_ptr(tokens), z_out.data_ptr(), _ptr(hdraft_out), _stream_ptr(stream))
        B.check(rc, "outlets_predict_step_noalloc" if noalloc else "outlets_predict_step")
        return z_out[:n], (hdraft_out[:n] if hdraft_out is not None else None)

    def release(self, slots: Sequence[int]) -> None:
        B.check(B.outlets_release(self.ctx, list(slots)), "outlets_release")

    # ------------------------------------------------------------ MLP probe
    def probe_prefill(self, slots: Sequence[int], lens: Sequence[int], h: torch.Tensor,
                      row_stride: Optional[int] = None, z_out: Optional[torch.Tensor] = None, stream=None):
        n = len(slots)
        if z_out is None:
            z_out = torch.empty(max(n, 1), dtype=torch.float32, device=self.device)
        stride = h.stride(0) if row_stride is None else row_stride
        B.check(B.outlets_probe_prefill(self.ctx, list(slots), list(lens), h.data_ptr(), stride,
                                        z_out.data_ptr(), _stream_ptr(stream)), "outlets_probe_prefill")
        return z_out[:n]

    def probe_step(self, slots: Sequence[int], h: torch.Tensor, row_stride: Optional[int] = None,
                   z_out: Optional[torch.Tensor] = None, stream=None):
        n = len(slots)
        if z_out is None:
            z_out = torch.empty(max(n, 1), dtype=torch.float32, device=self.device)
        stride = h.stride(0) if row_stride is None else row_stride
        B.check(B.outlets_probe_step(self.ctx, list(slots), h.data_ptr(), stride, z_out.data_ptr(),
                                     _stream_ptr(stream)), "outlets_probe_step")
        return z_out[:n]

    def probe_release(self, slots: Sequence[int]) -> None:
        B.check(B.outlets_probe_release(self.ctx, list(slots)), "outlets_probe_release")

    # ------------------------------------------------------------ draft model head
    def draft_distribution(self, n_req: int, p_out: Optional[torch.Tensor] = None, stream=None):
        """Eq. 2 for the requests of the last prefill/step call: [n_req, V] fp32."""
        if p_out is None:
            p_out = torch.empty((max(n_req, 1), self.vocab), dtype=torch.float32, device=self.device)
        B.check(B.outlets_draft_distribution(self.ctx, n_req, p_out.data_ptr(), _stream_ptr(stream)),
                "outlets_draft_distribution")
        return p_out[:n_req]

    # ------------------------------------------------------------ inspection
    def profile(self, enable: bool, groups=None) -> None:
        """Time every kernel group (or only the named ones, e.g. ["ATTN"]) of
        later calls; enable=False stops."""
        if groups is None:
            B.outlets_profile_enable(self.ctx, enable)
        else:
            mask = sum(1 << B.KERNELS.index(g) for g in groups) if enable else 0
            B.outlets_profile_enable_groups(self.ctx, mask)

    def profile_read(self, call: str = "prefill"):
        """{kernel group: (total ms, launches)} of prefill or step calls since
        profiling was enabled."""
        c = {"prefill": 0, "step": 1}[call]
        return {name: B.outlets_profile_read(self.ctx, c, i) for i, name in enumerate(B.KERNELS)}

    def meta(self, what: int):
        cap = self.cfg.max_slots * (-(-self.cfg.max_seq_len // 16)) + self.cfg.max_batch_tokens + 1
        return np.array(B.outlets_get_meta(self.ctx, what, cap), dtype=np.int32)

    def buffer(self, name: str, dtype: torch.dtype) -> torch.Tensor:
        which = B.BUF[name]
        nbytes = B.outlets_buffer_size(self.ctx, which)
        out = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=self.device)
        B.outlets_get_buffer(self.ctx, which, out.data_ptr(), nbytes, _stream_ptr(None))
        torch.cuda.synchronize(self.device)
        return out[:nbytes].view(dtype)

    def close(self):
        if getattr(self, "ctx", None):
            torch.cuda.synchronize(self.device)
            B.outlets_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
