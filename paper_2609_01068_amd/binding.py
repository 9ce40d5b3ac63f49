"""ctypes binding of ``liboutlets.so`` (the C ABI declared in include/outlets.h).

Argument marshalling only: every step of the path runs in the HIP library.
Loading fails loudly when the library has not been built; there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
# OUTLETS_LIB may name another build of the same library (e.g. a tuning variant)
LIB_PATH = os.environ.get("OUTLETS_LIB") or os.path.join(PKG, "liboutlets.so")

OUTLETS_OK = 0
OUTLETS_ERR_INVALID_ARG = -1
OUTLETS_ERR_SLOT_BUSY = -2
OUTLETS_ERR_SLOT_EMPTY = -3
OUTLETS_ERR_OUT_OF_PAGES = -4
OUTLETS_ERR_UNSUPPORTED = -5
OUTLETS_ERR_HIP = -6
OUTLETS_ERR_NOMEM = -7

OUTLETS_FMT_F32 = 0
OUTLETS_FMT_BF16 = 1
OUTLETS_FMT_E4M3 = 2

OUTLETS_META_PAGE_TABLE = 0
OUTLETS_META_SEQ_LEN = 1
OUTLETS_META_DEV_PAGE_TABLE = 2
OUTLETS_META_DEV_CU_SEQLENS = 3
OUTLETS_META_DEV_POSITIONS = 4
OUTLETS_META_DEV_LAST_IDX = 5
OUTLETS_META_DEV_TOKEN_SLOT = 6

KERNELS = ["META", "FUSE_GEMM", "NORM", "QKV_GEMM", "ROPE_KV", "ATTN", "O_GEMM", "GATE_UP_GEMM",
           "DOWN_GEMM", "POOL", "HEAD"]

BUF = {name: i for i, name in enumerate(
    ["FUSED", "NORM_ATTN", "Q", "ATTN", "X1", "NORM_MLP", "MLP_ACT", "X2", "HDRAFT",
     "POOLED", "K_POOL", "V_POOL", "NORM_EMB"])}


class OutletsError(RuntimeError):
    def __init__(self, rc: int, fn: str, msg: str):
        super().__init__(f"{fn} failed with status {rc}: {msg}")
        self.rc = rc


class outlets_config(C.Structure):
    _fields_ = [
        ("d_model", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
        ("head_dim", C.c_int32), ("ffn_dim", C.c_int32), ("head_hidden", C.c_int32),
        ("rope_theta", C.c_double), ("rms_eps", C.c_float), ("weight_fmt", C.c_int32),
        ("act_fmt", C.c_int32), ("page_size", C.c_int32), ("max_slots", C.c_int32),
        ("max_seq_len", C.c_int32), ("num_pages", C.c_int32), ("max_batch_tokens", C.c_int32),
        ("max_batch_requests", C.c_int32), ("keep_intermediates", C.c_int32), ("vocab", C.c_int32),
    ]


WEIGHT_FIELDS = [
    "w_proj", "s_proj", "w_q", "s_q", "w_k", "s_k", "w_v", "s_v", "w_o", "s_o",
    "w_gate", "s_gate", "w_up", "s_up", "w_down", "s_down", "gamma_attn", "gamma_mlp",
    "gamma_final", "head_w1", "head_b1", "head_w2", "head_b2", "w_attn_gate", "s_attn_gate",
    "probe_w1", "probe_b1", "probe_w2", "probe_b2", "w_lm", "s_lm", "embed", "gamma_emb",
]


class outlets_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in WEIGHT_FIELDS]


OUTLETS_ROUTE_RR, OUTLETS_ROUTE_LB = 0, 1
OUTLETS_QUEUE_FCFS, OUTLETS_QUEUE_SJF = 0, 1


class outlets_sim_config(C.Structure):
    _fields_ = [("n_instances", C.c_int32), ("max_running", C.c_int32), ("routing", C.c_int32),
                ("queue_order", C.c_int32), ("iter_base_us", C.c_int64), ("iter_per_seq_us", C.c_int64)]


_lib: Optional[C.CDLL] = None

_P = C.c_void_p
_I32P = C.POINTER(C.c_int32)
_SIGS = {
    "outlets_create": (C.c_int, [C.POINTER(outlets_config), C.POINTER(outlets_weights), C.c_int32, C.POINTER(_P)]),
    "outlets_destroy": (C.c_int, [_P]),
    "outlets_predict_prefill": (C.c_int, [_P, C.c_int32, _I32P, _I32P, _P, _P, _P, C.c_int64, _P, _P, _P, _P]),
    "outlets_predict_step": (C.c_int, [_P, C.c_int32, _I32P, _P, _P, _P, C.c_int64, _P, _P, _P, _P]),
    "outlets_predict_step_noalloc": (C.c_int, [_P, C.c_int32, _I32P, _P, _P, _P, C.c_int64, _P, _P, _P, _P]),
    "outlets_release": (C.c_int, [_P, C.c_int32, _I32P]),
    "outlets_probe_prefill": (C.c_int, [_P, C.c_int32, _I32P, _I32P, _P, C.c_int64, _P, _P]),
    "outlets_probe_step": (C.c_int, [_P, C.c_int32, _I32P, _P, C.c_int64, _P, _P]),
    "outlets_probe_release": (C.c_int, [_P, C.c_int32, _I32P]),
    "outlets_draft_distribution": (C.c_int, [_P, C.c_int32, _P, _P]),
    "outlets_get_meta": (C.c_int, [_P, C.c_int32, _I32P, C.c_int64, C.POINTER(C.c_int64)]),
    "outlets_get_buffer": (C.c_int, [_P, C.c_int32, _P, C.c_int64, C.POINTER(C.c_int64), _P]),
    "outlets_last_error": (C.c_char_p, []),
    "outlets_profile_enable": (C.c_int, [_P, C.c_int32]),
    "outlets_profile_enable_groups": (C.c_int, [_P, C.c_uint32]),
    "outlets_profile_read": (C.c_int, [_P, C.c_int32, C.c_int32, C.POINTER(C.c_double), C.POINTER(C.c_int64)]),
    "outlets_varlen_meta": (C.c_int, [C.c_int32, _I32P, _I32P, _I32P, _I32P]),
    "outlets_decode_plan": (C.c_int, [C.c_int32, _I32P, C.c_int32, C.c_int32, _I32P, _I32P, C.c_int64, _I32P,
                                      _I32P, C.c_int64]),
    "outlets_pager_create": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.POINTER(_P)]),
    "outlets_pager_destroy": (C.c_int, [_P]),
    "outlets_pager_prefill": (C.c_int, [_P, C.c_int32, _I32P, _I32P]),
    "outlets_pager_step": (C.c_int, [_P, C.c_int32, _I32P]),
    "outlets_pager_release": (C.c_int, [_P, C.c_int32, _I32P]),
    "outlets_pager_read": (C.c_int, [_P, C.c_int32, _I32P, C.c_int64, C.POINTER(C.c_int64)]),
    "outlets_pred_tokens": (C.c_int, [C.c_int32, _P, _P]),
    "outlets_sched_create": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.POINTER(_P)]),
    "outlets_sched_destroy": (C.c_int, [_P]),
    "outlets_sched_submit": (C.c_int, [_P, C.c_int32, _I32P, _I32P, _I32P]),
    "outlets_sched_admit": (C.c_int, [_P, C.c_int32, C.c_int32, _I32P, _I32P]),
    "outlets_sched_iteration": (C.c_int, [_P, C.c_int32]),
    "outlets_sched_finish": (C.c_int, [_P, C.c_int32, _I32P]),
    "outlets_sched_read": (C.c_int, [_P, C.c_int32, C.POINTER(C.c_int64), _I32P, _I32P]),
    "outlets_sched_simulate": (C.c_int, [C.POINTER(outlets_sim_config), C.c_int32, _P, _P, _P, _P, _P, _P]),
    "outlets_sched_metrics": (C.c_int, [C.c_int32, _P, _P, _P, C.c_int32, C.c_int32, _P]),
}


def lib() -> C.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_01068_amd.build` (there is no fallback)")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def exported_names():
    return list(_SIGS)


def last_error() -> str:
    return lib().outlets_last_error().decode()


def check(rc: int, fn: str) -> int:
    if rc != OUTLETS_OK:
        raise OutletsError(rc, fn, last_error())
    return rc


def i32_array(values):
    vals = [int(v) for v in values]
    return (C.c_int32 * max(1, len(vals)))(*vals)


# ------------------------------------------------------------ thin wrappers

def outlets_create(cfg: outlets_config, weights: outlets_weights, device: int = 0) -> C.c_void_p:
    ctx = C.c_void_p()
    check(lib().outlets_create(C.byref(cfg), C.byref(weights), device, C.byref(ctx)), "outlets_create")
    return ctx


def outlets_destroy(ctx) -> None:
    lib().outlets_destroy(ctx)


def outlets_predict_prefill(ctx, slots, lens, h_low: int, h_mid: int, h_high: int, row_stride: int,
                            tokens: Optional[int], z_out: int, hdraft_out: Optional[int],
                            stream: Optional[int]) -> int:
    n = len(slots)
    return lib().outlets_predict_prefill(ctx, n, i32_array(slots), i32_array(lens), h_low, h_mid, h_high,
                                         row_stride, tokens, z_out, hdraft_out, stream)


def outlets_predict_step(ctx, slots, h_low: int, h_mid: int, h_high: int, row_stride: int,
                         tokens: Optional[int], z_out: int, hdraft_out: Optional[int],
                         stream: Optional[int]) -> int:
    return lib().outlets_predict_step(ctx, len(slots), i32_array(slots), h_low, h_mid, h_high, row_stride,
                                      tokens, z_out, hdraft_out, stream)


def outlets_predict_step_noalloc(ctx, slots, h_low: int, h_mid: int, h_high: int, row_stride: int,
                                 tokens: Optional[int], z_out: int, hdraft_out: Optional[int],
                                 stream: Optional[int]) -> int:
    return lib().outlets_predict_step_noalloc(ctx, len(slots), i32_array(slots), h_low, h_mid, h_high,
                                              row_stride, tokens, z_out, hdraft_out, stream)


def outlets_release(ctx, slots) -> int:
    return lib().outlets_release(ctx, len(slots), i32_array(slots))


def outlets_probe_prefill(ctx, slots, lens, h: int, row_stride: int, z_out: int,
                          stream: Optional[int]) -> int:
    return lib().outlets_probe_prefill(ctx, len(slots), i32_array(slots), i32_array(lens), h, row_stride,
                                       z_out, stream)


def outlets_probe_step(ctx, slots, h: int, row_stride: int, z_out: int, stream: Optional[int]) -> int:
    return lib().outlets_probe_step(ctx, len(slots), i32_array(slots), h, row_stride, z_out, stream)


def outlets_probe_release(ctx, slots) -> int:
    return lib().outlets_probe_release(ctx, len(slots), i32_array(slots))


def outlets_draft_distribution(ctx, n_req: int, p_out: int, stream: Optional[int]) -> int:
    return lib().outlets_draft_distribution(ctx, n_req, p_out, stream)


def outlets_get_meta(ctx, what: int, cap: int):
    buf = (C.c_int32 * max(1, cap))()
    n = C.c_int64()
    check(lib().outlets_get_meta(ctx, what, buf, cap, C.byref(n)), "outlets_get_meta")
    return list(buf[:n.value])


def outlets_get_buffer(ctx, which: int, dst: int, nbytes: int, stream: Optional[int]) -> int:
    n = C.c_int64()
    check(lib().outlets_get_buffer(ctx, which, dst, nbytes, C.byref(n), stream), "outlets_get_buffer")
    return n.value


def outlets_buffer_size(ctx, which: int) -> int:
    n = C.c_int64()
    lib().outlets_get_buffer(ctx, which, None, 0, C.byref(n), None)
    return n.value


def outlets_profile_enable(ctx, enable: bool) -> None:
    check(lib().outlets_profile_enable(ctx, int(bool(enable))), "outlets_profile_enable")


def outlets_profile_enable_groups(ctx, groups: int) -> None:
    check(lib().outlets_profile_enable_groups(ctx, int(groups) & 0xFFFFFFFF), "outlets_profile_enable_groups")


def outlets_profile_read(ctx, call: int, which: int):
    ms, n = C.c_double(), C.c_int64()
    check(lib().outlets_profile_read(ctx, call, which, C.byref(ms), C.byref(n)), "outlets_profile_read")
    return ms.value, n.value


def outlets_varlen_meta(lens):
    n = len(lens)
    T = int(sum(int(x) for x in lens))
    cu, pos, last = (C.c_int32 * (n + 1))(), (C.c_int32 * max(1, T))(), (C.c_int32 * max(1, n))()
    check(lib().outlets_varlen_meta(n, i32_array(lens), cu, pos, last), "outlets_varlen_meta")
    return list(cu), list(pos[:T]), list(last[:n])


def outlets_decode_plan(pages, n_kv: int, cus: int):
    """The decode-attention work plan of a step (host only): returns
    (work [n_pieces, 4] rows of (request, first page, end page, segment),
    cu_segs [n_req + 1], lane_off [n_lanes + 1])."""
    n = len(pages)
    pg = i32_array(pages)
    counts = (C.c_int32 * 3)()
    check(lib().outlets_decode_plan(n, pg, n_kv, cus, counts, None, 0, None, None, 0), "outlets_decode_plan")
    n_pieces, n_segs, n_lanes = list(counts)
    work, cu, lanes = (C.c_int32 * (4 * n_pieces))(), (C.c_int32 * (n + 1))(), (C.c_int32 * (n_lanes + 1))()
    check(lib().outlets_decode_plan(n, pg, n_kv, cus, counts, work, 4 * n_pieces, cu, lanes, n_lanes + 1),
          "outlets_decode_plan")
    return [tuple(work[4 * i:4 * i + 4]) for i in range(n_pieces)], list(cu), list(lanes)


class Pager:
    """Host-only page allocator of the library (no GPU involved)."""

    def __init__(self, num_pages: int, page_size: int, max_slots: int, max_seq_len: int):
        self.h = C.c_void_p()
        check(lib().outlets_pager_create(num_pages, page_size, max_slots, max_seq_len, C.byref(self.h)),
              "outlets_pager_create")
        self.max_slots = max_slots
        self.max_pages = -(-max_seq_len // page_size)

    def prefill(self, slots, lens) -> int:
        return lib().outlets_pager_prefill(self.h, len(slots), i32_array(slots), i32_array(lens))

    def step(self, slots) -> int:
        return lib().outlets_pager_step(self.h, len(slots), i32_array(slots))

    def release(self, slots) -> int:
        return lib().outlets_pager_release(self.h, len(slots), i32_array(slots))

    def read(self, what: int):
        cap = self.max_slots * self.max_pages
        buf = (C.c_int32 * cap)()
        n = C.c_int64()
        check(lib().outlets_pager_read(self.h, what, buf, cap, C.byref(n)), "outlets_pager_read")
        return list(buf[:n.value])

    def close(self):
        if self.h:
            lib().outlets_pager_destroy(self.h)
            self.h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ------------------------------------------------------------ control plane (host only)

def _np(a, dtype):
    import numpy as np
    return np.ascontiguousarray(a, dtype=dtype)


def outlets_pred_tokens(z_hat):
    """Whole-token predicted lengths from z_hat (host floats)."""
    import numpy as np
    z = _np(z_hat, np.float32)
    out = np.empty(len(z), dtype=np.int32)
    check(lib().outlets_pred_tokens(len(z), z.ctypes.data, out.ctypes.data), "outlets_pred_tokens")
    return out


def outlets_sched_simulate(arrival_us, out_len, pred_tokens, n_instances: int, max_running: int,
                           routing: int, queue_order: int, iter_base_us: int, iter_per_seq_us: int):
    """Run the decode-cluster simulation; returns (instance, start_us, finish_us) arrays."""
    import numpy as np
    a, L, p = _np(arrival_us, np.int64), _np(out_len, np.int32), _np(pred_tokens, np.int32)
    n = len(a)
    if len(L) != n or len(p) != n:
        raise ValueError("trace arrays differ in length")
    cfg = outlets_sim_config(n_instances, max_running, routing, queue_order, iter_base_us, iter_per_seq_us)
    inst = np.full(n, -1, dtype=np.int32)
    start = np.full(n, -1, dtype=np.int64)
    finish = np.full(n, -1, dtype=np.int64)
    check(lib().outlets_sched_simulate(C.byref(cfg), n, a.ctypes.data, L.ctypes.data, p.ctypes.data,
                                       inst.ctypes.data, start.ctypes.data, finish.ctypes.data),
          "outlets_sched_simulate")
    return inst, start, finish


def outlets_sched_metrics(arrival_us, out_len, finish_us, short_below: int = 800, long_from: int = 1300):
    """(tokens/s, mean latency s, P99 short, P99 medium, P99 long, makespan s)."""
    import numpy as np
    a, L, f = _np(arrival_us, np.int64), _np(out_len, np.int32), _np(finish_us, np.int64)
    out = np.empty(6, dtype=np.float64)
    check(lib().outlets_sched_metrics(len(a), a.ctypes.data, L.ctypes.data, f.ctypes.data, short_below,
                                      long_from, out.ctypes.data), "outlets_sched_metrics")
    return tuple(float(x) for x in out)


class ControlPlane:
    """The library's online control plane (host only)."""

    def __init__(self, n_instances: int, max_running: int, routing: int, queue_order: int, max_requests: int):
        self.h = C.c_void_p()
        check(lib().outlets_sched_create(n_instances, max_running, routing, queue_order, max_requests,
                                         C.byref(self.h)), "outlets_sched_create")
        self.max_running = max_running

    def submit(self, ids, preds):
        out = (C.c_int32 * max(1, len(ids)))()
        check(lib().outlets_sched_submit(self.h, len(ids), i32_array(ids), i32_array(preds), out),
              "outlets_sched_submit")
        return list(out[:len(ids)])

    def admit(self, instance: int, cap: Optional[int] = None):
        cap = self.max_running if cap is None else cap
        out = (C.c_int32 * max(1, cap))()
        n = C.c_int32()
        check(lib().outlets_sched_admit(self.h, instance, cap, out, C.byref(n)), "outlets_sched_admit")
        return list(out[:n.value])

    def iteration(self, instance: int) -> None:
        check(lib().outlets_sched_iteration(self.h, instance), "outlets_sched_iteration")

    def finish(self, ids) -> None:
        check(lib().outlets_sched_finish(self.h, len(ids), i32_array(ids)), "outlets_sched_finish")

    def read(self, instance: int):
        load, w, r = C.c_int64(), C.c_int32(), C.c_int32()
        check(lib().outlets_sched_read(self.h, instance, C.byref(load), C.byref(w), C.byref(r)),
              "outlets_sched_read")
        return load.value, w.value, r.value

    def close(self):
        if self.h:
            lib().outlets_sched_destroy(self.h)
            self.h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
