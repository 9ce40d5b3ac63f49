// C ABI of the library: context set-up, the two prediction calls, slot
// release and inspection.  Host work per call is validation, page allocation
// (Pager), and one pinned host->device copy of the call's request metadata
// and page-table updates; everything else is kernels queued on the caller's
// stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "kernels.hpp"
#include "outlets.h"
#include "pager.hpp"
#include "sched.hpp"

using namespace outlets;

namespace {

thread_local std::string g_err;

int fail(int rc, const std::string& msg) {
    g_err = msg;
    return rc;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(OUTLETS_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                              \
    do {                                                 \
        hipError_t e_ = (expr);                          \
        if (e_ != hipSuccess) return hip_fail(e_, what); \
    } while (0)

size_t fmt_bytes(int fmt) { return fmt == FMT_F32 ? 4 : (fmt == FMT_BF16 ? 2 : 1); }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

constexpr int kHeadSplits = 8;      // K splits of the length head GEMM (at least)

}  // namespace

// Static scratch of outlets_predict_step_noalloc: one decode step's per-call
// buffers for callers that cannot allocate device memory.  Each device that
// loads the library holds its own copy until the process ends; every
// no-allocation step on that device works in it, so such calls must not
// overlap on one device.  Host code never passes `scratch` itself to a
// kernel (in host code it names a host-side stand-in): it uses the device
// address hipGetSymbolAddress returns, looked up once per device.
static constexpr size_t kScratchBytes = static_cast<size_t>(256) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};   // device address of `scratch`, per device

}  // namespace

// Device buffers a predict call works in: activations, partial sums and the
// call's metadata.  The context owns one set (sized at create for its
// capacities); outlets_predict_step_noalloc lays another set over the
// library's static scratch array.
struct CallBufs {
    float* r_f = nullptr;   // residual stream: f_ctx, x1, x2, h_draft (aliases unless kept)
    float* r_x1 = nullptr;
    float* r_x2 = nullptr;
    float* r_h = nullptr;
    void* a_norm = nullptr;
    void* b_norm = nullptr;
    void* e_norm = nullptr;      // [T, d] act: RMSNorm(embed[token]) * gamma_emb
    void* qkv = nullptr;
    void* attn = nullptr;
    void* mlp = nullptr;
    float* pooled = nullptr;
    uint16_t* pooled_bf16 = nullptr;
    float* head_part = nullptr;
    int32_t* tok_slot = nullptr;
    int32_t* tok_pos = nullptr;
    int32_t* last_idx = nullptr;
    int32_t* d_meta = nullptr;   // req_off | req_slot | req_start | page updates | work list
    int64_t meta_cap = 0;        // int32 entries
    float* pool_part = nullptr;  // [max tiles, d] prefill pooling partial sums
    float* decode_part = nullptr;  // split-KV decode attention partials
    float* splitk_ws = nullptr;  // fp32 partial sums of split-K GEMMs
    size_t splitk_bytes = 0;
};

struct outlets_ctx {
    outlets_config cfg{};
    outlets_weights w{};
    int device = 0;
    int act_fmt = 0, w_fmt = 0, small_fmt = 0;  // small_fmt: gains and head
    int64_t d = 0, qdim = 0, kvdim = 0, qkv_dim = 0, F = 0, H1 = 0;
    bool gated = false;          // Gated Attention: q|k|v|g rows, output gate in attention
    bool probe = false;          // MLP probe weights present
    bool embed_in = false;       // EAGLE-3 input embeddings: attention reads [emb ; norm(f)] (2d)
    int64_t k_attn = 0;          // width of the attention block's input row: d or 2d
    std::vector<int32_t> probe_count;   // per slot: tokens pooled by the probe (0 = inactive)
    float* probe_sum = nullptr;  // [max_slots, d] running sums of the probe's input rows
    int32_t* probe_meta = nullptr;   // req_off | req_slot | req_start | cu_tiles of a probe call
    float* lm_logits = nullptr;  // draft model head logits [2 * max_batch_requests, V]
    float* lm_stats = nullptr;   // draft model head softmax: per-chunk max and sum
    std::unique_ptr<Pager> pager;
    int max_pages = 0;

    std::vector<void*> allocs;
    CallBufs cb;                 // the context's own per-call buffers
    void* kpool = nullptr;
    void* vpool = nullptr;
    int32_t* page_table = nullptr;
    float* pool_sum = nullptr;
    float* cos_t = nullptr;
    float* sin_t = nullptr;

    int64_t work_off = 0;        // offset of the prefill attention work list in d_meta
    int32_t n_work = 0;
    int32_t attn_qtile = 32;       // queries per prefill attention work item of the current call
    int64_t tiles_off = 0;       // offset of cu_tiles (prefill pooling) in d_meta
    int64_t lanes_off = 0;       // offset of the decode plan's range offsets in d_meta
    int32_t n_lanes = 0;         // decode page ranges (waves per KV head) of the current call
    int32_t n_tiles = 0;

    int32_t* h_stage[2] = {nullptr, nullptr};
    hipEvent_t ev[2] = {nullptr, nullptr};
    bool ev_used[2] = {false, false};
    int stage = 0;

    int32_t last_n = 0, last_T = 0;
    bool last_in_scratch = false;   // the last predict call ran in the static scratch
    void* scratch = nullptr;        // this device's address of the static scratch

    // per-kernel timing (outlets_profile_enable)
    bool prof_on = false;
    uint32_t prof_mask = 0;   // kernel groups timed while prof_on
    struct Mark { int phase, which; hipEvent_t a, b; };
    std::vector<Mark> marks;
    std::vector<hipEvent_t> spare;
    int prof_phase = 0;                      // 0: prefill call, 1: step call
    double prof_ms[2][OUTLETS_K_COUNT] = {};
    int64_t prof_n[2][OUTLETS_K_COUNT] = {};

    ~outlets_ctx() {
        (void)hipSetDevice(device);
        (void)hipDeviceSynchronize();
        for (void* p : allocs) (void)hipFree(p);
        for (int i = 0; i < 2; ++i) {
            if (h_stage[i]) (void)hipHostFree(h_stage[i]);
            if (ev[i]) (void)hipEventDestroy(ev[i]);
        }
        for (auto& m : marks) { (void)hipEventDestroy(m.a); (void)hipEventDestroy(m.b); }
        for (auto e : spare) (void)hipEventDestroy(e);
    }

    hipEvent_t take_event() {
        hipEvent_t e = nullptr;
        if (!spare.empty()) { e = spare.back(); spare.pop_back(); return e; }
        // timing only: no system-scope fence (a cache write-back and
        // invalidate per record would perturb the work being timed)
        if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
        return e;
    }

    int alloc(void** p, size_t bytes) {
        if (bytes == 0) bytes = 256;
        hipError_t e = hipMalloc(p, bytes);
        if (e != hipSuccess) {
            *p = nullptr;
            return fail(OUTLETS_ERR_NOMEM, std::string("hipMalloc of ") + std::to_string(bytes) +
                                               " bytes failed: " + hipGetErrorString(e));
        }
        allocs.push_back(*p);
        return OUTLETS_OK;
    }
};

namespace {

// Records an event pair around the launches of one kernel group when
// profiling is on.
struct KTimer {
    outlets_ctx* c;
    int which;
    hipStream_t st;
    hipEvent_t a = nullptr;
    KTimer(outlets_ctx* c_, int w, hipStream_t s) : c(c_), which(w), st(s) {
        if (c->prof_on && ((c->prof_mask >> which) & 1u) && (a = c->take_event())) (void)hipEventRecord(a, st);
    }
    ~KTimer() {
        if (!a) return;
        hipEvent_t b = c->take_event();
        if (!b) { c->spare.push_back(a); return; }
        (void)hipEventRecord(b, st);
        c->marks.push_back({c->prof_phase, which, a, b});
    }
};

void collect_marks(outlets_ctx* c) {
    for (auto& m : c->marks) {
        float ms = 0.f;
        if (hipEventSynchronize(m.b) == hipSuccess && hipEventElapsedTime(&ms, m.a, m.b) == hipSuccess) {
            c->prof_ms[m.phase][m.which] += ms;
            c->prof_n[m.phase][m.which] += 1;
        }
        c->spare.push_back(m.a);
        c->spare.push_back(m.b);
    }
    c->marks.clear();
}

// Device address of the static scratch on `device` (the current device),
// looked up once per device and kept.
int scratch_address(int device, void** out) {
    if (device < 0 || device >= kMaxDevices) return fail(OUTLETS_ERR_UNSUPPORTED, "device index above 63");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[device]) {
        void* p = nullptr;
        HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
        if (!p) return fail(OUTLETS_ERR_HIP, "hipGetSymbolAddress(scratch) returned null");
        g_scratch_dev[device] = p;
    }
    *out = g_scratch_dev[device];
    return OUTLETS_OK;
}

int check_config(const outlets_config& c, const char** why) {
    auto bad = [&](int rc, const char* msg) { *why = msg; return rc; };
    if (c.d_model <= 0 || c.n_q_heads <= 0 || c.n_kv_heads <= 0 || c.ffn_dim <= 0 || c.head_hidden <= 0)
        return bad(OUTLETS_ERR_INVALID_ARG, "dimensions must be positive");
    if (c.max_slots <= 0 || c.max_seq_len <= 0 || c.num_pages <= 0 || c.max_batch_tokens <= 0 ||
        c.max_batch_requests <= 0)
        return bad(OUTLETS_ERR_INVALID_ARG, "capacities must be positive");
    if (!(c.rms_eps >= 0.f) || !(c.rope_theta > 0.0))
        return bad(OUTLETS_ERR_INVALID_ARG, "rms_eps must be >= 0 and rope_theta > 0");
    if (!attn_supported(c.n_q_heads, c.n_kv_heads, c.head_dim))
        return bad(OUTLETS_ERR_UNSUPPORTED, "attention supports head_dim 64/128 and n_q/n_kv in {1,2,4,8}");
    if (c.page_size != 16) return bad(OUTLETS_ERR_UNSUPPORTED, "page_size must be 16");
    if (c.weight_fmt < 0 || c.weight_fmt > 2 || c.act_fmt < 0 || c.act_fmt > 1)
        return bad(OUTLETS_ERR_UNSUPPORTED, "unknown weight or activation format");
    if (c.weight_fmt == OUTLETS_FMT_F32 && c.act_fmt != OUTLETS_FMT_F32)
        return bad(OUTLETS_ERR_UNSUPPORTED, "f32 weights need f32 activations");
    if (c.weight_fmt != OUTLETS_FMT_F32 && c.act_fmt != OUTLETS_FMT_BF16)
        return bad(OUTLETS_ERR_UNSUPPORTED, "bf16/e4m3 weights need bf16 activations");
    if (c.vocab < 0) return bad(OUTLETS_ERR_INVALID_ARG, "vocab must be >= 0");
    *why = nullptr;
    return OUTLETS_OK;
}

GemmA gemm_a(const void* p, int64_t ld, int64_t kseg) {
    GemmA a{};
    a.p[0] = p;
    a.ld = ld;
    a.kseg = static_cast<int32_t>(kseg);
    return a;
}

GemmB gemm_b1(const void* p, const void* scale, int64_t rows, int64_t ld) {
    GemmB b{};
    b.p[0] = p;
    b.scale[0] = static_cast<const uint16_t*>(scale);
    b.nend[0] = b.nend[1] = b.nend[2] = b.nend[3] = static_cast<int32_t>(rows);
    b.ld = ld;
    return b;
}

GemmC gemm_c(void* c, int64_t ldc, const float* resid = nullptr, int64_t ldr = 0) {
    GemmC r{};
    r.c = c;
    r.ldc = ldc;
    r.resid = resid;
    r.ldr = ldr;
    return r;
}

// The per-layer GEMM descriptors; M varies per call.
struct LayerGemms {
    GemmA a_fuse, a_qkv, a_o, a_gu, a_down, a_head;
    GemmB b_fuse, b_qkv, b_o, b_gu, b_down, b_head;
    int64_t n_gu;
};

LayerGemms layer_gemms(const outlets_ctx* c, const CallBufs& b, const void* hl, const void* hm, const void* hh,
                       int64_t row_stride) {
    LayerGemms g{};
    const auto& w = c->w;
    const int64_t d = c->d;
    g.a_fuse = gemm_a(hl, row_stride, d);
    g.a_fuse.p[1] = hm;
    g.a_fuse.p[2] = hh;
    g.b_fuse = gemm_b1(w.w_proj, w.s_proj, d, 3 * d);
    if (c->embed_in) {
        // input embeddings: K = 2d over [normed embedding | normed f_ctx]
        g.a_qkv = gemm_a(b.e_norm, d, d);
        g.a_qkv.p[1] = b.a_norm;
    } else {
        g.a_qkv = gemm_a(b.a_norm, d, d);
    }
    g.b_qkv = gemm_b1(w.w_q, w.s_q, c->qdim, c->k_attn);
    g.b_qkv.p[1] = w.w_k;
    g.b_qkv.p[2] = w.w_v;
    g.b_qkv.scale[1] = static_cast<const uint16_t*>(w.s_k);
    g.b_qkv.scale[2] = static_cast<const uint16_t*>(w.s_v);
    g.b_qkv.nend[0] = static_cast<int32_t>(c->qdim);
    g.b_qkv.nend[1] = static_cast<int32_t>(c->qdim + c->kvdim);
    g.b_qkv.nend[2] = static_cast<int32_t>(c->qdim + 2 * c->kvdim);
    g.b_qkv.nend[3] = static_cast<int32_t>(c->qkv_dim);
    if (c->gated) {
        // Gated Attention: the gate projection is a fourth row segment
        g.b_qkv.p[3] = w.w_attn_gate;
        g.b_qkv.scale[3] = static_cast<const uint16_t*>(w.s_attn_gate);
    }
    g.a_o = gemm_a(b.attn, c->qdim, c->qdim);
    g.b_o = gemm_b1(w.w_o, w.s_o, d, c->qdim);
    g.a_gu = gemm_a(b.b_norm, d, d);
    g.b_gu = gemm_b1(w.w_gate, w.s_gate, c->F, d);
    g.b_gu.p[1] = w.w_up;
    g.b_gu.scale[1] = static_cast<const uint16_t*>(w.s_up);
    if (c->w_fmt == FMT_F32) {
        g.n_gu = c->F;            // dual-row VALU kernel
    } else {
        g.b_gu.paired = 1;        // 32-row gate/up interleave
        g.n_gu = 2 * c->F;
    }
    g.a_down = gemm_a(b.mlp, c->F, c->F);
    g.b_down = gemm_b1(w.w_down, w.s_down, d, c->F);
    if (c->w_fmt == FMT_F32)
        g.a_head = gemm_a(b.pooled, 2 * d, 2 * d);
    else
        g.a_head = gemm_a(b.pooled_bf16, 2 * d, 2 * d);
    g.b_head = gemm_b1(w.head_w1, nullptr, c->H1, 2 * d);
    return g;
}

// Draft model head input: the newest token's h_draft is the second half of
// each pooled row ([mean ; newest]); bf16 weights read its hi/lo split.
// K splits of the head GEMM over `rows` A rows: kHeadSplits, doubled up to
// 32 while the workgroups fill at most half the CUs and every split keeps at
// least 4 K slices of 64 (the fp32 path keeps kHeadSplits).  Measured: 32
// splits for 64 rows take the head from 0.033 to 0.024 ms; 16 instead of 8
// for 1,024 rows is slower (the finish reads twice the partials).
int head_splits(const outlets_ctx* c, int rows) {
    int s = kHeadSplits;
    if (c->w_fmt == FMT_F32) return s;
    const int tiles = ((rows + 255) / 256) * static_cast<int>((c->H1 + 255) / 256);
    const int kslices = static_cast<int>(2 * c->d / 64);
    while (s < 32 && tiles * 2 * s <= gemm_device_cus() / 2 && kslices / (2 * s) >= 4) s *= 2;
    return s;
}

GemmA lm_input(const outlets_ctx* c) {
    return (c->w_fmt == FMT_F32) ? gemm_a(c->cb.pooled + c->d, 2 * c->d, c->d)
                                 : gemm_a(c->cb.pooled_bf16 + c->d, 2 * c->d, c->d);
}

int check_gemms(const outlets_ctx* c) {
    // Dummy 16-byte aligned pointers stand in for the per-call A operands.
    LayerGemms g = layer_gemms(c, c->cb, c->cb.a_norm, c->cb.a_norm, c->cb.a_norm, c->d);
    const char* why = nullptr;
    const int af = c->act_fmt, wf = c->w_fmt;
    const int hf = (wf == FMT_F32) ? FMT_F32 : FMT_BF16;
    int rc;
    if ((rc = gemm_check(af, wf, EPI_STORE_F32, 1, c->d, 3 * c->d, g.a_fuse, g.b_fuse, 1, &why)) ||
        (rc = gemm_check(af, wf, EPI_STORE_ACT, 1, c->qkv_dim, c->k_attn, g.a_qkv, g.b_qkv, 1, &why)) ||
        (rc = gemm_check(af, wf, EPI_RESID_F32, 1, c->d, c->qdim, g.a_o, g.b_o, 1, &why)) ||
        (rc = gemm_check(af, wf, EPI_SWIGLU, 1, g.n_gu, c->d, g.a_gu, g.b_gu, 1, &why)) ||
        (rc = gemm_check(af, wf, EPI_RESID_F32, 1, c->d, c->F, g.a_down, g.b_down, 1, &why)) ||
        (rc = gemm_check(af, hf, EPI_PARTIAL, 1, c->H1, 2 * c->d, g.a_head, g.b_head, kHeadSplits, &why)))
        return fail(rc, std::string("unsupported shape: ") + why);
    if (c->w.w_lm) {
        const GemmA a = lm_input(c);
        const GemmB b = gemm_b1(c->w.w_lm, c->w.s_lm, c->cfg.vocab, c->d);
        if ((rc = gemm_check(af, wf, EPI_STORE_F32, 1, c->cfg.vocab, c->d, a, b, 1, &why)))
            return fail(rc, std::string("unsupported draft head shape: ") + why);
    }
    return OUTLETS_OK;
}

// Queue the draft layer + head for `T` tokens of `n` requests whose
// metadata is already on the device.
int run_layer(outlets_ctx* c, const CallBufs& b, bool prefill, int n, int T, const void* hl, const void* hm,
              const void* hh, int64_t row_stride, const int32_t* tokens, float* z_out,
              void* hdraft_out, hipStream_t st) {
    const int af = c->act_fmt, wf = c->w_fmt;
    const int64_t d = c->d;
    LayerGemms g = layer_gemms(c, b, hl, hm, hh, row_stride);
    const int32_t* req_off = b.d_meta;
    const int32_t* req_slot = b.d_meta + (n + 1);
    const int32_t* req_start = b.d_meta + (n + 1) + n;
    const float eps = c->cfg.rms_eps;

    // A GEMM whose K is split (small M) followed by an RMSNorm leaves its
    // partial sums to the norm kernel, which adds them (and the residual),
    // stores the residual-stream row and normalises it in one pass.
    auto fusable = [&](const void* gamma) {
        return wf != FMT_F32 && rowsum_supported(static_cast<int>(d)) && aligned16(gamma);
    };
    auto rowsum = [&](int S, const float* resid, float* out) {
        return RowSum{b.splitk_ws, S, static_cast<int64_t>(T) * d, d, resid, d, out, d};
    };
    // Eq. 1: f_ctx = W_proj [h_low | h_mid | h_high]
    int sk = 0;
    { KTimer t(c, OUTLETS_K_FUSE_GEMM, st);
      if (fusable(c->w.gamma_attn))
          sk = gemm_launch_partials(af, wf, EPI_STORE_F32, T, d, 3 * d, g.a_fuse, g.b_fuse, b.splitk_ws,
                                    b.splitk_bytes, st);
      if (!sk)
          gemm_launch(af, wf, EPI_STORE_F32, T, d, 3 * d, g.a_fuse, g.b_fuse, gemm_c(b.r_f, d), 1, st, b.splitk_ws,
                      b.splitk_bytes); }
    { KTimer t(c, OUTLETS_K_NORM, st);
      if (sk)
          launch_rmsnorm_sum(af, c->small_fmt, T, d, rowsum(sk, nullptr, b.r_f), c->w.gamma_attn, eps, b.a_norm, d,
                             st);
      else
          launch_rmsnorm(af, c->small_fmt, T, d, b.r_f, d, c->w.gamma_attn, eps, b.a_norm, d, nullptr, 0, st);
      if (c->embed_in)
          launch_embed_norm(af, c->small_fmt, T, static_cast<int>(d), c->cfg.vocab, tokens, c->w.embed,
                            c->w.gamma_emb, eps, b.e_norm, d, st); }
    // QKV projection; with bf16 activations and head dim 128, RoPE and the
    // paged K/V write happen in its epilogue (or in its split-K reduce)
    if (gemm_qkv_rope_fusable(af, wf, c->cfg.n_q_heads, c->cfg.n_kv_heads, c->cfg.head_dim,
                              static_cast<int>(c->qkv_dim))) {
        KTimer t(c, OUTLETS_K_QKV_GEMM, st);
        GemmC qc = gemm_c(b.qkv, c->qkv_dim);
        qc.rope = RopeKV{b.tok_pos, b.tok_slot, c->page_table, static_cast<int32_t>(c->max_pages),
                         c->cfg.n_q_heads, c->cfg.n_kv_heads, static_cast<uint16_t*>(c->kpool),
                         static_cast<uint16_t*>(c->vpool), c->cos_t, c->sin_t};
        gemm_launch(af, wf, EPI_QKV_ROPE, T, c->qkv_dim, static_cast<int>(c->k_attn), g.a_qkv, g.b_qkv, qc, 1, st,
                    b.splitk_ws, b.splitk_bytes);
    } else {
        { KTimer t(c, OUTLETS_K_QKV_GEMM, st);
          gemm_launch(af, wf, EPI_STORE_ACT, T, c->qkv_dim, static_cast<int>(c->k_attn), g.a_qkv, g.b_qkv, gemm_c(b.qkv, c->qkv_dim), 1, st, b.splitk_ws, b.splitk_bytes); }
        { KTimer t(c, OUTLETS_K_ROPE_KV, st);
          launch_rope_kv(af, T, b.qkv, c->qkv_dim, b.tok_slot, b.tok_pos, c->page_table, c->max_pages,
                         c->kpool, c->vpool, c->cos_t, c->sin_t, c->cfg.n_q_heads, c->cfg.n_kv_heads,
                         c->cfg.head_dim, st); }
    }
    { KTimer t(c, OUTLETS_K_ATTN, st);
      const void* gate = c->gated ? static_cast<const char*>(b.qkv) + (c->qdim + 2 * c->kvdim) * fmt_bytes(af)
                                  : nullptr;
      if (prefill && c->n_work > 0)
          launch_attn_prefill(c->n_work, b.d_meta + c->work_off, c->attn_qtile, b.qkv, c->qkv_dim, b.attn, c->qdim,
                              req_off, req_slot, c->page_table, c->max_pages, c->kpool, c->vpool,
                              c->cfg.n_q_heads, c->cfg.n_kv_heads, gate, st);
      else if (!prefill && c->n_work > 0)
          launch_attn_decode(n, c->n_work, b.d_meta + c->work_off, b.d_meta + c->tiles_off,
                             c->n_lanes, b.d_meta + c->lanes_off, b.qkv,
                             c->qkv_dim, b.attn, c->qdim, req_slot, req_start, c->page_table,
                             c->max_pages, c->kpool, c->vpool, c->cfg.n_q_heads, c->cfg.n_kv_heads,
                             b.decode_part, gate, st);
      else
          launch_attn_paged(af, T, b.qkv, c->qkv_dim, b.attn, c->qdim, b.tok_slot, b.tok_pos,
                            c->page_table, c->max_pages, c->kpool, c->vpool, c->cfg.n_q_heads,
                            c->cfg.n_kv_heads, c->cfg.head_dim, gate, st); }
    sk = 0;
    { KTimer t(c, OUTLETS_K_O_GEMM, st);
      if (fusable(c->w.gamma_mlp))
          sk = gemm_launch_partials(af, wf, EPI_RESID_F32, T, d, c->qdim, g.a_o, g.b_o, b.splitk_ws, b.splitk_bytes,
                                    st);
      if (!sk)
          gemm_launch(af, wf, EPI_RESID_F32, T, d, c->qdim, g.a_o, g.b_o, gemm_c(b.r_x1, d, b.r_f, d), 1, st,
                      b.splitk_ws, b.splitk_bytes); }
    { KTimer t(c, OUTLETS_K_NORM, st);
      if (sk)
          launch_rmsnorm_sum(af, c->small_fmt, T, d, rowsum(sk, b.r_f, b.r_x1), c->w.gamma_mlp, eps, b.b_norm, d,
                             st);
      else
          launch_rmsnorm(af, c->small_fmt, T, d, b.r_x1, d, c->w.gamma_mlp, eps, b.b_norm, d, nullptr, 0, st); }
    { KTimer t(c, OUTLETS_K_GATE_UP_GEMM, st);
      gemm_launch(af, wf, EPI_SWIGLU, T, g.n_gu, d, g.a_gu, g.b_gu, gemm_c(b.mlp, c->F), 1, st, b.splitk_ws, b.splitk_bytes); }
    // steps: the down GEMM's partials go to the final norm + pooling kernel
    sk = 0;
    { KTimer t(c, OUTLETS_K_DOWN_GEMM, st);
      if (!prefill && fusable(c->w.gamma_final))
          sk = gemm_launch_partials(af, wf, EPI_RESID_F32, T, d, c->F, g.a_down, g.b_down, b.splitk_ws,
                                    b.splitk_bytes, st);
      if (!sk)
          gemm_launch(af, wf, EPI_RESID_F32, T, d, c->F, g.a_down, g.b_down, gemm_c(b.r_x2, d, b.r_x1, d), 1, st,
                      b.splitk_ws, b.splitk_bytes); }
    const RowSum down_rows = rowsum(sk, b.r_x1, c->cfg.keep_intermediates ? b.r_x2 : nullptr);
    uint16_t* pb = (wf == FMT_F32) ? nullptr : b.pooled_bf16;
    // prefill: final RMSNorm + pooling in one pass over x2 (h_draft rows are
    // stored only when the caller wants them or intermediates are kept; the
    // pooling needs only each request's last row)
    bool fused_pool = false;
    if (prefill) {
        KTimer t(c, OUTLETS_K_POOL, st);
        fused_pool = launch_norm_pool_prefill(
            af, c->small_fmt, n, c->n_tiles, d, b.r_x2, d, c->w.gamma_final, eps, hdraft_out, d, b.r_h, d,
            hdraft_out != nullptr || c->cfg.keep_intermediates != 0, req_off, req_slot, b.d_meta + c->tiles_off,
            b.pool_part, c->pool_sum, b.pooled, pb, st);
    } else {
        // steps (one row per request): the f32 h_draft rows are kept only
        // with intermediates
        KTimer t(c, OUTLETS_K_POOL, st);
        fused_pool = launch_norm_pool_step(af, c->small_fmt, n, d, sk ? nullptr : b.r_x2, d, c->w.gamma_final, eps,
                                           hdraft_out, d, c->cfg.keep_intermediates ? b.r_h : nullptr, d, req_slot,
                                           req_start, c->pool_sum, b.pooled, pb, st, sk ? &down_rows : nullptr);
        if (sk && !fused_pool) return fail(OUTLETS_ERR_HIP, "internal: split down GEMM without its norm kernel");
    }
    if (!fused_pool) {
        { KTimer t(c, OUTLETS_K_NORM, st);
          launch_rmsnorm(af, c->small_fmt, T, d, b.r_x2, d, c->w.gamma_final, eps, hdraft_out, d, b.r_h, d, st); }
        { KTimer t(c, OUTLETS_K_POOL, st);
          if (prefill)
              launch_pool_prefill(n, c->n_tiles, d, FMT_F32, b.r_h, d, req_off, req_slot, b.d_meta + c->tiles_off,
                                  b.pool_part, c->pool_sum, b.pooled, pb, st);
          else
              launch_pool_step(n, d, FMT_F32, b.r_h, d, req_slot, req_start, c->pool_sum, b.pooled, pb, st); }
    }
    const int hf = (wf == FMT_F32) ? FMT_F32 : FMT_BF16;
    // bf16 heads read the hi/lo split of the pooled vector: 2n rows
    const int head_rows = (wf == FMT_F32) ? n : 2 * n;
    GemmC hc = gemm_c(b.head_part, c->H1);
    hc.split_stride = static_cast<int64_t>(head_rows) * c->H1;
    const int hs = head_splits(c, head_rows);
    { KTimer t(c, OUTLETS_K_HEAD, st);
      gemm_launch(af, hf, EPI_PARTIAL, head_rows, c->H1, 2 * d, g.a_head, g.b_head, hc, hs, st);
      launch_head_finish(c->small_fmt, n, c->H1, hs, b.head_part, c->w.head_b1, c->w.head_w2,
                         c->w.head_b2, z_out, st); }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return OUTLETS_OK;
}

// Stage req_off | req_slot | req_start | updates into pinned memory and copy to the device.
int upload_meta(outlets_ctx* c, const CallBufs& b, int n, const std::vector<int32_t>& off, const int32_t* slots,
                const std::vector<int32_t>& start, const std::vector<int32_t>& updates,
                const std::vector<int32_t>& work, const std::vector<int32_t>& cu_tiles,
                const std::vector<int32_t>& lanes, int work_stride, hipStream_t st) {
    const int64_t count = (n + 1) + 2 * static_cast<int64_t>(n) + static_cast<int64_t>(updates.size()) +
                          static_cast<int64_t>(work.size()) + static_cast<int64_t>(cu_tiles.size()) +
                          static_cast<int64_t>(lanes.size());
    if (count > b.meta_cap) return fail(OUTLETS_ERR_INVALID_ARG, "call metadata exceeds capacity");
    const int s = c->stage;
    if (c->ev_used[s]) HIP_TRY(hipEventSynchronize(c->ev[s]), "hipEventSynchronize");
    int32_t* h = c->h_stage[s];
    std::memcpy(h, off.data(), sizeof(int32_t) * (n + 1));
    std::memcpy(h + n + 1, slots, sizeof(int32_t) * n);
    std::memcpy(h + 2 * n + 1, start.data(), sizeof(int32_t) * n);
    if (!updates.empty()) std::memcpy(h + 3 * n + 1, updates.data(), sizeof(int32_t) * updates.size());
    c->work_off = 3 * n + 1 + static_cast<int64_t>(updates.size());
    c->n_work = static_cast<int32_t>(work.size() / work_stride);
    if (!work.empty()) std::memcpy(h + c->work_off, work.data(), sizeof(int32_t) * work.size());
    c->tiles_off = c->work_off + static_cast<int64_t>(work.size());
    c->n_tiles = cu_tiles.empty() ? 0 : cu_tiles.back();
    if (!cu_tiles.empty()) std::memcpy(h + c->tiles_off, cu_tiles.data(), sizeof(int32_t) * cu_tiles.size());
    c->lanes_off = c->tiles_off + static_cast<int64_t>(cu_tiles.size());
    if (!lanes.empty()) std::memcpy(h + c->lanes_off, lanes.data(), sizeof(int32_t) * lanes.size());
    {
        // one kernel reads the staged block from host memory (no copy-engine
        // transfer on the call's critical path), applies the page-table
        // updates and builds the token arrays
        KTimer t(c, OUTLETS_K_META, st);
        launch_meta_fetch(h, static_cast<int>(count), n, static_cast<int>(updates.size() / 2), b.d_meta,
                          c->page_table, b.tok_slot, b.tok_pos, b.last_idx, st);
    }
    HIP_TRY(hipEventRecord(c->ev[s], st), "hipEventRecord");
    c->ev_used[s] = true;
    c->stage ^= 1;
    return OUTLETS_OK;
}

// Prefill attention work items (request, tile of qt queries), longest
// first: a tile's cost is the number of 64-key tiles it visits.
std::vector<int32_t> attention_work(int n, const int32_t* lens, int qt) {
    std::vector<std::pair<int32_t, int32_t>> items;
    for (int i = 0; i < n; ++i)
        for (int t = 0; t * qt < lens[i]; ++t) items.emplace_back(i, t);
    auto cost = [&](const std::pair<int32_t, int32_t>& it) {
        return std::min(it.second * qt + qt - 1, lens[it.first] - 1) / 64;
    };
    std::stable_sort(items.begin(), items.end(),
                     [&](const auto& a, const auto& b) { return cost(a) > cost(b); });
    std::vector<int32_t> out;
    out.reserve(2 * items.size());
    for (auto& it : items) { out.push_back(it.first); out.push_back(it.second); }
    return out;
}

int check_states(const outlets_ctx* c, const void* hl, const void* hm, const void* hh,
                 int64_t row_stride, const int32_t* tokens, const float* z_out) {
    if (!hl || !hm || !hh || !z_out) return fail(OUTLETS_ERR_INVALID_ARG, "null state or output pointer");
    if (c->embed_in && !tokens) return fail(OUTLETS_ERR_INVALID_ARG, "input embeddings need token ids");
    if (row_stride < c->d) return fail(OUTLETS_ERR_INVALID_ARG, "row_stride < d_model");
    if (c->act_fmt == FMT_BF16 && (row_stride % 8 || !aligned16(hl) || !aligned16(hm) || !aligned16(hh)))
        return fail(OUTLETS_ERR_UNSUPPORTED, "bf16 states need 16-byte aligned rows (row_stride % 8 == 0)");
    return OUTLETS_OK;
}

// ---------------------------------------------------------------- decode steps

// Buffers of a decode step of n requests laid over `base` (256-byte aligned
// pieces): metadata (meta_count int32), token arrays, activations, pooled
// rows, and one region shared by the split-K workspace (ws_bytes), the
// split-KV attention partials and the head partials, whose uses are ordered
// one after another on the call's stream.  With base == nullptr only the
// size is computed.  Returns the bytes used.
size_t layout_step(const outlets_ctx* c, int n, int64_t n_records, int64_t meta_count, size_t ws_bytes,
                   char* base, CallBufs* b) {
    size_t off = 0;
    auto take = [&](size_t bytes) -> char* {
        off = (off + 255) & ~static_cast<size_t>(255);
        char* p = base ? base + off : nullptr;
        off += bytes;
        return p;
    };
    const size_t ab = fmt_bytes(c->act_fmt);
    const size_t N = static_cast<size_t>(n);
    *b = CallBufs{};
    b->meta_cap = meta_count;
    b->d_meta = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * meta_count));
    b->tok_slot = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * N));
    b->tok_pos = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * N));
    b->last_idx = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * N));
    b->r_f = b->r_x1 = b->r_x2 = b->r_h = reinterpret_cast<float*>(take(sizeof(float) * N * c->d));
    b->a_norm = b->b_norm = take(ab * N * c->d);
    if (c->embed_in) b->e_norm = take(ab * N * c->d);
    b->qkv = take(ab * N * c->qkv_dim);
    b->attn = take(ab * N * c->qdim);
    b->mlp = take(ab * N * c->F);
    b->pooled = reinterpret_cast<float*>(take(sizeof(float) * N * 2 * c->d));
    if (c->w_fmt != FMT_F32) b->pooled_bf16 = reinterpret_cast<uint16_t*>(take(sizeof(uint16_t) * 2 * N * 2 * c->d));
    size_t region = ws_bytes;
    if (attn_prefill_mfma_supported(c->act_fmt, c->cfg.n_q_heads, c->cfg.n_kv_heads, c->cfg.head_dim))
        region = std::max(region, sizeof(float) * static_cast<size_t>(n_records) * c->cfg.n_q_heads *
                                      attn_decode_record_floats());
    const int rows = (c->w_fmt == FMT_F32 ? 1 : 2) * n;
    region = std::max(region, sizeof(float) * static_cast<size_t>(head_splits(c, rows)) * rows * c->H1);
    char* shared = take(region);
    b->splitk_ws = b->decode_part = b->head_part = reinterpret_cast<float*>(shared);
    b->splitk_bytes = ws_bytes;
    return off;
}

// Split-K workspace the layer's GEMMs use at M rows with the context's own
// workspace capacity (so a step in the static scratch takes the same plans,
// and gives the same results, as one in the context's buffers).
size_t step_splitk_bytes(const outlets_ctx* c, int M) {
    const int qkv_epi = gemm_qkv_rope_fusable(c->act_fmt, c->w_fmt, c->cfg.n_q_heads, c->cfg.n_kv_heads,
                                              c->cfg.head_dim, static_cast<int>(c->qkv_dim))
                            ? EPI_QKV_ROPE : EPI_STORE_ACT;
    const int64_t n_gu = (c->w_fmt == FMT_F32) ? c->F : 2 * c->F;
    const int64_t nk[5][2] = {{c->d, 3 * c->d}, {c->qkv_dim, c->k_attn}, {c->d, c->qdim}, {n_gu, c->d}, {c->d, c->F}};
    const int epis[5] = {EPI_STORE_F32, qkv_epi, EPI_RESID_F32, EPI_SWIGLU, EPI_RESID_F32};
    size_t need = 0;
    for (int g = 0; g < 5; ++g)
        need = std::max(need, gemm_workspace_bytes(c->w_fmt, epis[g], M, static_cast<int>(nk[g][0]),
                                                   static_cast<int>(nk[g][1]), c->cb.splitk_bytes));
    return need;
}

// Suspends per-kernel timing for one call (event creation is an allocation).
struct NoTiming {
    outlets_ctx* c;
    bool was;
    explicit NoTiming(outlets_ctx* c_, bool on) : c(c_), was(c_->prof_on) { if (on) c->prof_on = false; }
    ~NoTiming() { c->prof_on = was; }
};

// Dynamic prediction (Section 3.2, t >= 1) in the context's buffers or, with
// noalloc, in the static scratch array.
int predict_step_impl(outlets_ctx* ctx, bool noalloc, int32_t n_req, const int32_t* slots, const void* h_low,
                      const void* h_mid, const void* h_high, int64_t row_stride, const int32_t* tokens,
                      float* z_out, void* hdraft_out, void* stream) {
    if (!ctx) return fail(OUTLETS_ERR_INVALID_ARG, "null context");
    if (n_req < 0 || n_req > ctx->cfg.max_batch_requests || n_req > ctx->cfg.max_batch_tokens)
        return fail(OUTLETS_ERR_INVALID_ARG, "n_req outside [0, max_batch_requests]");
    if (noalloc && ctx->cfg.keep_intermediates)
        return fail(OUTLETS_ERR_UNSUPPORTED, "the no-allocation step does not keep intermediates");
    if (noalloc && !ctx->scratch) return fail(OUTLETS_ERR_HIP, "static scratch address unknown on this device");
    if (n_req == 0) return OUTLETS_OK;
    if (!slots) return fail(OUTLETS_ERR_INVALID_ARG, "null slots");
    int rc = check_states(ctx, h_low, h_mid, h_high, row_stride, tokens, z_out);
    if (rc) return rc;
    if (hdraft_out && ctx->act_fmt == FMT_BF16 && !aligned16(hdraft_out))
        return fail(OUTLETS_ERR_UNSUPPORTED, "hdraft_out must be 16-byte aligned");
    const char* why = "";
    rc = ctx->pager->check_step(n_req, slots, &why);
    if (rc) return fail(rc, why);
    HIP_TRY(hipSetDevice(ctx->device), "hipSetDevice");
    hipStream_t st = static_cast<hipStream_t>(stream);

    // the new token's position is each slot's cached length before the append
    std::vector<int32_t> off(n_req + 1), start(n_req);
    for (int i = 0; i <= n_req; ++i) off[i] = i;
    int32_t new_pages = 0;
    for (int i = 0; i < n_req; ++i) {
        start[i] = ctx->pager->seq_len(slots[i]);
        new_pages += (start[i] % 16 == 0);
    }
    // split-KV decode: the step's pages cut into equal contiguous ranges, one
    // per wave and KV head (segments and pieces, see attn_decode_plan)
    DecodePlan plan;
    if (attn_prefill_mfma_supported(ctx->act_fmt, ctx->cfg.n_q_heads, ctx->cfg.n_kv_heads, ctx->cfg.head_dim)) {
        std::vector<int32_t> pages(n_req);
        for (int i = 0; i < n_req; ++i) pages[i] = (start[i] + 1 + 15) / 16;
        attn_decode_plan(n_req, pages.data(), ctx->cfg.n_kv_heads, gemm_device_cus(), &plan);
    }
    CallBufs sb;
    const CallBufs* bufs = &ctx->cb;
    if (noalloc) {
        const int64_t n_records = plan.n_segs;
        const int64_t meta_count = (n_req + 1) + 2 * static_cast<int64_t>(n_req) + 2 * new_pages +
                                   static_cast<int64_t>(plan.work.size() + plan.cu_segs.size() + plan.lanes.size());
        const size_t ws = step_splitk_bytes(ctx, n_req);
        const size_t need = layout_step(ctx, n_req, n_records, meta_count, ws, nullptr, &sb);
        if (need > kScratchBytes)
            return fail(OUTLETS_ERR_INVALID_ARG, "the step needs " + std::to_string(need) +
                                                     " bytes of scratch; the static scratch holds " +
                                                     std::to_string(kScratchBytes));
        layout_step(ctx, n_req, n_records, meta_count, ws, static_cast<char*>(ctx->scratch), &sb);
        bufs = &sb;
    }
    std::vector<int32_t> updates;
    ctx->prof_phase = 1;
    rc = ctx->pager->step(n_req, slots, &updates, &why);
    if (rc) return fail(rc, why);
    ctx->n_lanes = plan.n_lanes;
    NoTiming nt(ctx, noalloc);
    rc = upload_meta(ctx, *bufs, n_req, off, slots, start, updates, plan.work, plan.cu_segs, plan.lanes, 4, st);
    if (rc == OUTLETS_OK)
        rc = run_layer(ctx, *bufs, false, n_req, n_req, h_low, h_mid, h_high, row_stride, tokens, z_out,
                       hdraft_out, st);
    if (rc) return rc;   // device work may be partly queued; the slot lengths advanced
    ctx->last_n = n_req;
    ctx->last_T = n_req;
    ctx->last_in_scratch = noalloc;
    return OUTLETS_OK;
}

}  // namespace

extern "C" {

const char* outlets_last_error(void) { return g_err.c_str(); }

int outlets_create(const outlets_config* cfg, const outlets_weights* weights, int32_t device,
                   outlets_ctx** out) {
    if (!out) return fail(OUTLETS_ERR_INVALID_ARG, "out is null");
    *out = nullptr;
    if (!cfg || !weights) return fail(OUTLETS_ERR_INVALID_ARG, "null config or weights");
    const char* why = nullptr;
    int rc = check_config(*cfg, &why);
    if (rc) return fail(rc, std::string("config: ") + why);
    const outlets_weights& w = *weights;
    const void* req[] = {w.w_proj, w.w_q, w.w_k, w.w_v, w.w_o, w.w_gate, w.w_up, w.w_down,
                         w.gamma_attn, w.gamma_mlp, w.gamma_final, w.head_w1, w.head_b1,
                         w.head_w2, w.head_b2};
    for (const void* p : req)
        if (!p) return fail(OUTLETS_ERR_INVALID_ARG, "a weight pointer is null");
    if ((w.embed != nullptr) != (w.gamma_emb != nullptr))
        return fail(OUTLETS_ERR_INVALID_ARG, "input embeddings need embed and gamma_emb");
    if ((cfg->vocab > 0) != (w.w_lm != nullptr || w.embed != nullptr))
        return fail(OUTLETS_ERR_INVALID_ARG, "vocab > 0 exactly when w_lm or embed is given");
    if (w.w_lm && cfg->weight_fmt == OUTLETS_FMT_E4M3 && !w.s_lm)
        return fail(OUTLETS_ERR_INVALID_ARG, "e4m3 weights need every row-scale pointer");
    if (w.w_lm && cfg->weight_fmt != OUTLETS_FMT_F32 && cfg->vocab % 256)
        return fail(OUTLETS_ERR_UNSUPPORTED, "bf16/e4m3 draft heads need vocab a multiple of 256");
    if (w.probe_w1 && (!w.probe_b1 || !w.probe_w2 || !w.probe_b2))
        return fail(OUTLETS_ERR_INVALID_ARG, "probe weights need w1, b1, w2 and b2");
    if (cfg->weight_fmt == OUTLETS_FMT_E4M3) {
        const void* sc[] = {w.s_proj, w.s_q, w.s_k, w.s_v, w.s_o, w.s_gate, w.s_up, w.s_down};
        for (const void* p : sc)
            if (!p) return fail(OUTLETS_ERR_INVALID_ARG, "e4m3 weights need every row-scale pointer");
        if (w.w_attn_gate && !w.s_attn_gate)
            return fail(OUTLETS_ERR_INVALID_ARG, "e4m3 weights need every row-scale pointer");
    }
    HIP_TRY(hipSetDevice(device), "hipSetDevice");
    void* scratch_ptr = nullptr;
    if ((rc = scratch_address(device, &scratch_ptr)) != OUTLETS_OK) return rc;

    std::unique_ptr<outlets_ctx> c;
    try {
        c.reset(new outlets_ctx());
        c->pager.reset(new Pager(cfg->num_pages, cfg->page_size, cfg->max_slots, cfg->max_seq_len));
    } catch (const std::bad_alloc&) {
        return fail(OUTLETS_ERR_NOMEM, "host allocation failed");
    }
    c->cfg = *cfg;
    c->w = w;
    c->device = device;
    c->scratch = scratch_ptr;
    c->act_fmt = cfg->act_fmt;
    c->w_fmt = cfg->weight_fmt;
    c->small_fmt = (cfg->weight_fmt == OUTLETS_FMT_F32) ? FMT_F32 : FMT_BF16;
    c->d = cfg->d_model;
    c->qdim = static_cast<int64_t>(cfg->n_q_heads) * cfg->head_dim;
    c->kvdim = static_cast<int64_t>(cfg->n_kv_heads) * cfg->head_dim;
    c->gated = w.w_attn_gate != nullptr;
    c->probe = w.probe_w1 != nullptr;
    c->qkv_dim = c->qdim + 2 * c->kvdim + (c->gated ? c->qdim : 0);
    c->embed_in = w.embed != nullptr;
    c->k_attn = (c->embed_in ? 2 : 1) * c->d;
    c->F = cfg->ffn_dim;
    c->H1 = cfg->head_hidden;
    c->max_pages = c->pager->max_pages_per_seq();

    const size_t ab = fmt_bytes(c->act_fmt);
    const int64_t Tm = cfg->max_batch_tokens, Bm = std::max(cfg->max_batch_requests, 1);
    const int64_t hd = cfg->head_dim;
    const size_t pool_elems = static_cast<size_t>(cfg->num_pages) * cfg->n_kv_heads * 16 * hd;
    void* p = nullptr;
#define ALLOC(dst, bytes)                                              \
    do {                                                               \
        if ((rc = c->alloc(&p, (bytes))) != OUTLETS_OK) return rc;     \
        dst = decltype(dst)(p);                                        \
    } while (0)
    ALLOC(c->kpool, pool_elems * ab);
    ALLOC(c->vpool, pool_elems * ab);
    ALLOC(c->page_table, sizeof(int32_t) * c->pager->table().size());
    ALLOC(c->pool_sum, sizeof(float) * cfg->max_slots * c->d);
    ALLOC(c->cos_t, sizeof(float) * cfg->max_seq_len * (hd / 2));
    ALLOC(c->sin_t, sizeof(float) * cfg->max_seq_len * (hd / 2));
    const bool keep = cfg->keep_intermediates != 0;
    ALLOC(c->cb.r_f, sizeof(float) * Tm * c->d);
    if (keep) {
        ALLOC(c->cb.r_x1, sizeof(float) * Tm * c->d);
        ALLOC(c->cb.r_x2, sizeof(float) * Tm * c->d);
        ALLOC(c->cb.r_h, sizeof(float) * Tm * c->d);
    } else {
        c->cb.r_x1 = c->cb.r_x2 = c->cb.r_h = c->cb.r_f;
    }
    ALLOC(c->cb.a_norm, ab * Tm * c->d);
    if (c->embed_in) ALLOC(c->cb.e_norm, ab * Tm * c->d);
    if (keep) ALLOC(c->cb.b_norm, ab * Tm * c->d);
    else c->cb.b_norm = c->cb.a_norm;
    ALLOC(c->cb.qkv, ab * Tm * c->qkv_dim);
    ALLOC(c->cb.attn, ab * Tm * c->qdim);
    ALLOC(c->cb.mlp, ab * Tm * c->F);
    ALLOC(c->cb.pooled, sizeof(float) * Bm * 2 * c->d);
    ALLOC(c->cb.pooled_bf16, sizeof(uint16_t) * 2 * Bm * 2 * c->d);
    {
        // head partials: the largest splits x rows over every batch size
        int64_t most = 0;
        for (int64_t b = 1; b <= Bm; ++b) {
            const int rows = static_cast<int>((c->w_fmt == FMT_F32 ? 1 : 2) * b);
            most = std::max<int64_t>(most, static_cast<int64_t>(head_splits(c.get(), rows)) * rows);
        }
        ALLOC(c->cb.head_part, sizeof(float) * most * c->H1);
    }
    ALLOC(c->cb.tok_slot, sizeof(int32_t) * Tm);
    ALLOC(c->cb.tok_pos, sizeof(int32_t) * Tm);
    ALLOC(c->cb.last_idx, sizeof(int32_t) * Bm);
    // decode plan bounds: segments (partial records) and pieces of a step
    const int64_t max_segs = attn_decode_max_segments(Bm, cfg->n_kv_heads, gemm_device_cus());
    const int64_t max_pieces = attn_decode_max_pieces(Bm, c->max_pages, cfg->n_kv_heads, gemm_device_cus());
    // req_off | req_slot | req_start | page updates | work list (prefill
    // tiles, 2 ints each, or decode pieces, 4 ints each) | cu tiles or
    // segments | decode lane offsets (at most one lane per segment)
    c->cb.meta_cap = 3 * Bm + 1 + 2 * (Tm / 16 + Bm) + std::max(2 * (Tm / 32 + Bm), 4 * max_pieces) + (Bm + 1) +
                     (max_segs + 1);
    if (attn_prefill_mfma_supported(c->act_fmt, cfg->n_q_heads, cfg->n_kv_heads, cfg->head_dim))
        ALLOC(c->cb.decode_part, sizeof(float) * max_segs * cfg->n_q_heads * attn_decode_record_floats());
    ALLOC(c->cb.pool_part, sizeof(float) * (Tm / 32 + Bm) * c->d);
    {
        // split-K scratch: the largest plan over the layer's GEMMs for M up to 1024
        const int64_t gemm_nk[5][2] = {{c->d, 3 * c->d}, {c->qkv_dim, c->k_attn}, {c->d, c->qdim},
                                       {(c->w_fmt == FMT_F32 ? 1 : 2) * c->F, c->d}, {c->d, c->F}};
        const int epis[5] = {EPI_STORE_F32, EPI_STORE_ACT, EPI_RESID_F32, EPI_SWIGLU, EPI_RESID_F32};
        size_t need = 0;
        for (int64_t m0 = 16; m0 <= 1024 && m0 - 16 < Tm; m0 += 16) {
            const int64_t m = std::min<int64_t>(m0, Tm);
            for (int g = 0; g < 5; ++g) {
                const int sk = gemm_splitk_plan(c->w_fmt, epis[g], (int)m, (int)gemm_nk[g][0], (int)gemm_nk[g][1]);
                if (sk > 1) need = std::max(need, (size_t)sk * m * gemm_nk[g][0] * sizeof(float));
            }
        }
        // large GEMMs split their last round of tiles over K: up to one
        // 256 x 256 fp32 block per CU (256 CUs)
        if (Tm > 256) need = std::max(need, (size_t)256 * 65536 * sizeof(float));
        c->cb.splitk_bytes = need;
        if (need) ALLOC(c->cb.splitk_ws, need);
    }
    ALLOC(c->cb.d_meta, sizeof(int32_t) * c->cb.meta_cap);
    if (w.w_lm) ALLOC(c->lm_logits, sizeof(float) * 2 * Bm * cfg->vocab);
    if (w.w_lm) ALLOC(c->lm_stats, sizeof(float) * lm_softmax_stats_floats(Bm));
    if (c->probe) {
        ALLOC(c->probe_sum, sizeof(float) * cfg->max_slots * c->d);
        ALLOC(c->probe_meta, sizeof(int32_t) * c->cb.meta_cap);
        c->probe_count.assign(cfg->max_slots, 0);
    }
#undef ALLOC
    for (int i = 0; i < 2; ++i) {
        // host-coherent: the metadata kernel reads it in place
        HIP_TRY(hipHostMalloc(reinterpret_cast<void**>(&c->h_stage[i]), sizeof(int32_t) * c->cb.meta_cap,
                              hipHostMallocCoherent),
                "hipHostMalloc");
        HIP_TRY(hipEventCreateWithFlags(&c->ev[i], hipEventDisableTiming), "hipEventCreate");
    }
    if ((rc = check_gemms(c.get())) != OUTLETS_OK) return rc;

    // RoPE tables: angle p * theta^(-2c/hd) evaluated in float64, stored float32.
    {
        const int64_t half = hd / 2;
        std::vector<float> cs(static_cast<size_t>(cfg->max_seq_len) * half), sn(cs.size());
        for (int64_t pos = 0; pos < cfg->max_seq_len; ++pos)
            for (int64_t ch = 0; ch < half; ++ch) {
                const double ang = static_cast<double>(pos) *
                                   std::pow(cfg->rope_theta, -2.0 * static_cast<double>(ch) / static_cast<double>(hd));
                cs[pos * half + ch] = static_cast<float>(std::cos(ang));
                sn[pos * half + ch] = static_cast<float>(std::sin(ang));
            }
        HIP_TRY(hipMemcpy(c->cos_t, cs.data(), sizeof(float) * cs.size(), hipMemcpyHostToDevice), "hipMemcpy");
        HIP_TRY(hipMemcpy(c->sin_t, sn.data(), sizeof(float) * sn.size(), hipMemcpyHostToDevice), "hipMemcpy");
    }
    HIP_TRY(hipMemset(c->page_table, 0xFF, sizeof(int32_t) * c->pager->table().size()), "hipMemset");
    HIP_TRY(hipMemset(c->pool_sum, 0, sizeof(float) * cfg->max_slots * c->d), "hipMemset");
    if (c->probe) HIP_TRY(hipMemset(c->probe_sum, 0, sizeof(float) * cfg->max_slots * c->d), "hipMemset");
    // attention kernels may read (and give zero weight to) rows of a page no
    // token has written yet: start from zeros so those rows are finite
    HIP_TRY(hipMemset(c->kpool, 0, pool_elems * ab), "hipMemset");
    HIP_TRY(hipMemset(c->vpool, 0, pool_elems * ab), "hipMemset");
    HIP_TRY(hipDeviceSynchronize(), "hipDeviceSynchronize");
    *out = c.release();
    return OUTLETS_OK;
}

int outlets_destroy(outlets_ctx* ctx) {
    delete ctx;
    return OUTLETS_OK;
}

int outlets_predict_prefill(outlets_ctx* ctx, int32_t n_req, const int32_t* slots,
                            const int32_t* lens, const void* h_low, const void* h_mid,
                            const void* h_high, int64_t row_stride, const int32_t* tokens,
                            float* z_out, void* hdraft_out, void* stream) {
    if (!ctx) return fail(OUTLETS_ERR_INVALID_ARG, "null context");
    if (n_req < 0 || n_req > ctx->cfg.max_batch_requests)
        return fail(OUTLETS_ERR_INVALID_ARG, "n_req outside [0, max_batch_requests]");
    if (n_req == 0) return OUTLETS_OK;
    if (!slots || !lens) return fail(OUTLETS_ERR_INVALID_ARG, "null slots or lens");
    int rc = check_states(ctx, h_low, h_mid, h_high, row_stride, tokens, z_out);
    if (rc) return rc;
    if (hdraft_out && ctx->act_fmt == FMT_BF16 && !aligned16(hdraft_out))
        return fail(OUTLETS_ERR_UNSUPPORTED, "hdraft_out must be 16-byte aligned");
    HIP_TRY(hipSetDevice(ctx->device), "hipSetDevice");
    hipStream_t st = static_cast<hipStream_t>(stream);

    std::vector<int32_t> updates;
    const char* why = "";
    ctx->prof_phase = 0;
    rc = ctx->pager->prefill(n_req, slots, lens, &updates, &why);
    if (rc) return fail(rc, why);
    std::vector<int32_t> off(n_req + 1), start(n_req, 0);
    int64_t T = 0;
    off[0] = 0;
    for (int i = 0; i < n_req; ++i) {
        T += lens[i];
        off[i + 1] = static_cast<int32_t>(std::min<int64_t>(T, INT32_MAX));
    }
    if (T > ctx->cfg.max_batch_tokens) {
        ctx->pager->release(n_req, slots, &why);   // undo: same free set as before
        return fail(OUTLETS_ERR_INVALID_ARG, "total prompt tokens exceed max_batch_tokens");
    }
    std::vector<int32_t> work;
    if (attn_prefill_mfma_supported(ctx->act_fmt, ctx->cfg.n_q_heads, ctx->cfg.n_kv_heads, ctx->cfg.head_dim)) {
        ctx->attn_qtile = attn_prefill_query_tile(ctx->cfg.n_q_heads, ctx->cfg.n_kv_heads, T, n_req);
        work = attention_work(n_req, lens, ctx->attn_qtile);
    }
    std::vector<int32_t> cu_tiles(n_req + 1, 0);
    for (int i = 0; i < n_req; ++i) cu_tiles[i + 1] = cu_tiles[i] + (lens[i] + 31) / 32;
    rc = upload_meta(ctx, ctx->cb, n_req, off, slots, start, updates, work, cu_tiles, {}, 2, st);
    if (rc == OUTLETS_OK)
        rc = run_layer(ctx, ctx->cb, true, n_req, static_cast<int>(T), h_low, h_mid, h_high, row_stride, tokens,
                       z_out, hdraft_out, st);
    if (rc) {
        std::string msg = g_err;
        ctx->pager->release(n_req, slots, &why);
        return fail(rc, msg);
    }
    ctx->last_n = n_req;
    ctx->last_T = static_cast<int32_t>(T);
    ctx->last_in_scratch = false;
    return OUTLETS_OK;
}

int outlets_predict_step(outlets_ctx* ctx, int32_t n_req, const int32_t* slots, const void* h_low,
                         const void* h_mid, const void* h_high, int64_t row_stride,
                         const int32_t* tokens, float* z_out, void* hdraft_out, void* stream) {
    return predict_step_impl(ctx, false, n_req, slots, h_low, h_mid, h_high, row_stride, tokens, z_out,
                             hdraft_out, stream);
}

int outlets_predict_step_noalloc(outlets_ctx* ctx, int32_t n_req, const int32_t* slots, const void* h_low,
                                 const void* h_mid, const void* h_high, int64_t row_stride,
                                 const int32_t* tokens, float* z_out, void* hdraft_out, void* stream) {
    return predict_step_impl(ctx, true, n_req, slots, h_low, h_mid, h_high, row_stride, tokens, z_out,
                             hdraft_out, stream);
}

// ---------------------------------------------------------------- MLP probe
// The probe baseline: the length head's pooling and MLP applied directly to a
// target-model hidden state (no draft layer), with its own weights and
// per-slot running sums.

// Stage int32 metadata through the pinned double buffer into probe_meta (the
// metadata kernel in copy-only mode: no copy-engine transfer to wait on).
int upload_probe_meta(outlets_ctx* c, const std::vector<int32_t>& v, hipStream_t st) {
    if (static_cast<int64_t>(v.size()) > c->cb.meta_cap) return fail(OUTLETS_ERR_INVALID_ARG, "call metadata exceeds capacity");
    const int s = c->stage;
    if (c->ev_used[s]) HIP_TRY(hipEventSynchronize(c->ev[s]), "hipEventSynchronize");
    std::memcpy(c->h_stage[s], v.data(), sizeof(int32_t) * v.size());
    launch_meta_fetch(c->h_stage[s], static_cast<int>(v.size()), 0, 0, c->probe_meta, nullptr, nullptr, nullptr,
                      nullptr, st);
    HIP_TRY(hipEventRecord(c->ev[s], st), "hipEventRecord");
    c->ev_used[s] = true;
    c->stage ^= 1;
    return OUTLETS_OK;
}

// z_out[i] = probe MLP of pooled row i (pooled / pooled_bf16 already filled).
int run_probe_head(outlets_ctx* c, int n, float* z_out, hipStream_t st) {
    const int af = c->act_fmt, wf = c->w_fmt;
    const int hf = (wf == FMT_F32) ? FMT_F32 : FMT_BF16;
    const int64_t d = c->d;
    const GemmA a = (wf == FMT_F32) ? gemm_a(c->cb.pooled, 2 * d, 2 * d) : gemm_a(c->cb.pooled_bf16, 2 * d, 2 * d);
    const GemmB b = gemm_b1(c->w.probe_w1, nullptr, c->H1, 2 * d);
    const int rows = (wf == FMT_F32) ? n : 2 * n;
    GemmC hc = gemm_c(c->cb.head_part, c->H1);
    hc.split_stride = static_cast<int64_t>(rows) * c->H1;
    const int hs = head_splits(c, rows);
    gemm_launch(af, hf, EPI_PARTIAL, rows, c->H1, 2 * d, a, b, hc, hs, st);
    launch_head_finish(c->small_fmt, n, c->H1, hs, c->cb.head_part, c->w.probe_b1, c->w.probe_w2,
                       c->w.probe_b2, z_out, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return OUTLETS_OK;
}

int check_probe_call(const outlets_ctx* ctx, int32_t n_req, const int32_t* slots, const void* h,
                     int64_t row_stride, const float* z_out) {
    if (!ctx) return fail(OUTLETS_ERR_INVALID_ARG, "null context");
    if (!ctx->probe) return fail(OUTLETS_ERR_UNSUPPORTED, "the context was created without probe weights");
    if (n_req < 0 || n_req > ctx->cfg.max_batch_requests)
        return fail(OUTLETS_ERR_INVALID_ARG, "n_req outside [0, max_batch_requests]");
    if (n_req == 0) return OUTLETS_OK;
    if (!slots || !h || !z_out) return fail(OUTLETS_ERR_INVALID_ARG, "null slots, state or output pointer");
    if (row_stride < ctx->d) return fail(OUTLETS_ERR_INVALID_ARG, "row_stride < d_model");
    std::vector<char> seen(ctx->cfg.max_slots, 0);
    for (int i = 0; i < n_req; ++i) {
        if (slots[i] < 0 || slots[i] >= ctx->cfg.max_slots) return fail(OUTLETS_ERR_INVALID_ARG, "slot id out of range");
        if (seen[slots[i]]) return fail(OUTLETS_ERR_INVALID_ARG, "duplicate slot");
        seen[slots[i]] = 1;
    }
    return OUTLETS_OK;
}

int outlets_probe_prefill(outlets_ctx* ctx, int32_t n_req, const int32_t* slots, const int32_t* lens,
                          const void* h, int64_t row_stride, float* z_out, void* stream) {
    int rc = check_probe_call(ctx, n_req, slots, h, row_stride, z_out);
    if (rc || n_req == 0) return rc;
    if (!lens) return fail(OUTLETS_ERR_INVALID_ARG, "null lens");
    int64_t T = 0;
    for (int i = 0; i < n_req; ++i) {
        if (ctx->probe_count[slots[i]] != 0) return fail(OUTLETS_ERR_SLOT_BUSY, "probe slot already active");
        if (lens[i] <= 0) return fail(OUTLETS_ERR_INVALID_ARG, "prompt length must be >= 1");
        T += lens[i];
    }
    if (T > ctx->cfg.max_batch_tokens) return fail(OUTLETS_ERR_INVALID_ARG, "total prompt tokens exceed max_batch_tokens");
    HIP_TRY(hipSetDevice(ctx->device), "hipSetDevice");
    hipStream_t st = static_cast<hipStream_t>(stream);
    // req_off [n+1] | req_slot [n] | cu_tiles [n+1]
    std::vector<int32_t> v(3 * n_req + 2);
    int32_t* off = v.data();
    int32_t* sl = off + n_req + 1;
    int32_t* cu = sl + n_req;
    off[0] = cu[0] = 0;
    for (int i = 0; i < n_req; ++i) {
        off[i + 1] = off[i] + lens[i];
        sl[i] = slots[i];
        cu[i + 1] = cu[i] + (lens[i] + 31) / 32;
    }
    if ((rc = upload_probe_meta(ctx, v, st)) != OUTLETS_OK) return rc;
    const int32_t* d_off = ctx->probe_meta;
    launch_pool_prefill(n_req, cu[n_req], static_cast<int>(ctx->d), ctx->act_fmt, h, row_stride, d_off,
                        d_off + n_req + 1, d_off + 2 * n_req + 1, ctx->cb.pool_part, ctx->probe_sum, ctx->cb.pooled,
                        ctx->w_fmt == FMT_F32 ? nullptr : ctx->cb.pooled_bf16, st);
    if ((rc = run_probe_head(ctx, n_req, z_out, st)) != OUTLETS_OK) return rc;
    for (int i = 0; i < n_req; ++i) ctx->probe_count[slots[i]] = lens[i];
    return OUTLETS_OK;
}

int outlets_probe_step(outlets_ctx* ctx, int32_t n_req, const int32_t* slots, const void* h,
                       int64_t row_stride, float* z_out, void* stream) {
    int rc = check_probe_call(ctx, n_req, slots, h, row_stride, z_out);
    if (rc || n_req == 0) return rc;
    for (int i = 0; i < n_req; ++i)
        if (ctx->probe_count[slots[i]] == 0) return fail(OUTLETS_ERR_SLOT_EMPTY, "probe slot not active");
    HIP_TRY(hipSetDevice(ctx->device), "hipSetDevice");
    hipStream_t st = static_cast<hipStream_t>(stream);
    // req_slot [n] | req_start [n] (tokens pooled before this one)
    std::vector<int32_t> v(2 * n_req);
    for (int i = 0; i < n_req; ++i) {
        v[i] = slots[i];
        v[n_req + i] = ctx->probe_count[slots[i]];
    }
    if ((rc = upload_probe_meta(ctx, v, st)) != OUTLETS_OK) return rc;
    launch_pool_step(n_req, static_cast<int>(ctx->d), ctx->act_fmt, h, row_stride, ctx->probe_meta,
                     ctx->probe_meta + n_req, ctx->probe_sum, ctx->cb.pooled,
                     ctx->w_fmt == FMT_F32 ? nullptr : ctx->cb.pooled_bf16, st);
    if ((rc = run_probe_head(ctx, n_req, z_out, st)) != OUTLETS_OK) return rc;
    for (int i = 0; i < n_req; ++i) ctx->probe_count[slots[i]] += 1;
    return OUTLETS_OK;
}

int outlets_probe_release(outlets_ctx* ctx, int32_t n, const int32_t* slots) {
    if (!ctx) return fail(OUTLETS_ERR_INVALID_ARG, "null context");
    if (!ctx->probe) return fail(OUTLETS_ERR_UNSUPPORTED, "the context was created without probe weights");
    if (n < 0 || (n > 0 && !slots)) return fail(OUTLETS_ERR_INVALID_ARG, "bad slot list");
    for (int i = 0; i < n; ++i)
        if (slots[i] < 0 || slots[i] >= ctx->cfg.max_slots) return fail(OUTLETS_ERR_INVALID_ARG, "slot id out of range");
    std::vector<char> seen(ctx->cfg.max_slots, 0);
    for (int i = 0; i < n; ++i) {
        if (seen[slots[i]]) return fail(OUTLETS_ERR_INVALID_ARG, "duplicate slot");
        seen[slots[i]] = 1;
    }
    for (int i = 0; i < n; ++i) ctx->probe_count[slots[i]] = 0;
    return OUTLETS_OK;
}

int outlets_draft_distribution(outlets_ctx* ctx, int32_t n_req, float* p_out, void* stream) {
    if (!ctx) return fail(OUTLETS_ERR_INVALID_ARG, "null context");
    if (!ctx->w.w_lm) return fail(OUTLETS_ERR_UNSUPPORTED, "the context has no draft model head (no w_lm)");
    if (n_req <= 0 || n_req != ctx->last_n)
        return fail(OUTLETS_ERR_INVALID_ARG, "n_req must equal the last predict call's request count");
    if (!p_out) return fail(OUTLETS_ERR_INVALID_ARG, "null p_out");
    if (ctx->last_in_scratch)
        return fail(OUTLETS_ERR_INVALID_ARG, "the last predict call ran in the static scratch (no-allocation step)");
    HIP_TRY(hipSetDevice(ctx->device), "hipSetDevice");
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int V = ctx->cfg.vocab;
    const bool split = ctx->w_fmt != FMT_F32;          // hi rows [0, n), lo rows [n, 2n)
    const int rows = split ? 2 * n_req : n_req;
    gemm_launch(ctx->act_fmt, ctx->w_fmt, EPI_STORE_F32, rows, V, static_cast<int>(ctx->d), lm_input(ctx),
                gemm_b1(ctx->w.w_lm, ctx->w.s_lm, V, ctx->d), gemm_c(ctx->lm_logits, V), 1, st,
                ctx->cb.splitk_ws, ctx->cb.splitk_bytes);
    launch_lm_softmax(n_req, V, ctx->lm_logits, split, ctx->lm_stats, p_out, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return OUTLETS_OK;
}

int outlets_release(outlets_ctx* ctx, int32_t n, const int32_t* slots) {
    if (!ctx) return fail(OUTLETS_ERR_INVALID_ARG, "null context");
    if (n < 0 || (n > 0 && !slots)) return fail(OUTLETS_ERR_INVALID_ARG, "bad slot list");
    const char* why = "";
    int rc = ctx->pager->release(n, slots, &why);
    return rc ? fail(rc, why) : OUTLETS_OK;
}

int outlets_get_meta(outlets_ctx* ctx, int32_t what, int32_t* out, int64_t cap, int64_t* n_out) {
    if (!ctx || !out || !n_out) return fail(OUTLETS_ERR_INVALID_ARG, "null argument");
    const int64_t n = ctx->last_n, T = ctx->last_T;
    int64_t count = 0;
    const void* dev = nullptr;
    switch (what) {
        case OUTLETS_META_PAGE_TABLE: count = static_cast<int64_t>(ctx->pager->table().size()); break;
        case OUTLETS_META_SEQ_LEN: count = ctx->pager->max_slots(); break;
        case OUTLETS_META_DEV_PAGE_TABLE: count = static_cast<int64_t>(ctx->pager->table().size()); dev = ctx->page_table; break;
        case OUTLETS_META_DEV_CU_SEQLENS: count = n + 1; dev = ctx->cb.d_meta; break;
        case OUTLETS_META_DEV_POSITIONS: count = T; dev = ctx->cb.tok_pos; break;
        case OUTLETS_META_DEV_LAST_IDX: count = n; dev = ctx->cb.last_idx; break;
        case OUTLETS_META_DEV_TOKEN_SLOT: count = T; dev = ctx->cb.tok_slot; break;
        default: return fail(OUTLETS_ERR_INVALID_ARG, "unknown metadata id");
    }
    *n_out = count;
    if (cap < count) return fail(OUTLETS_ERR_INVALID_ARG, "output capacity too small");
    if (ctx->last_in_scratch && what >= OUTLETS_META_DEV_CU_SEQLENS)
        return fail(OUTLETS_ERR_INVALID_ARG, "the last predict call ran in the static scratch (no-allocation step)");
    if (!dev) {
        const auto& v = (what == OUTLETS_META_PAGE_TABLE) ? ctx->pager->table() : ctx->pager->seq_lens();
        std::memcpy(out, v.data(), sizeof(int32_t) * count);
        return OUTLETS_OK;
    }
    HIP_TRY(hipSetDevice(ctx->device), "hipSetDevice");
    HIP_TRY(hipDeviceSynchronize(), "hipDeviceSynchronize");
    if (count) HIP_TRY(hipMemcpy(out, dev, sizeof(int32_t) * count, hipMemcpyDeviceToHost), "hipMemcpy");
    return OUTLETS_OK;
}

int outlets_get_buffer(outlets_ctx* ctx, int32_t which, void* dst, int64_t nbytes, int64_t* n_bytes,
                       void* stream) {
    if (!ctx || !n_bytes) return fail(OUTLETS_ERR_INVALID_ARG, "null argument");
    const int64_t T = ctx->last_T, n = ctx->last_n, d = ctx->d;
    const int64_t ab = static_cast<int64_t>(fmt_bytes(ctx->act_fmt));
    const bool keep = ctx->cfg.keep_intermediates != 0;
    const void* src = nullptr;
    int64_t size = 0;
    bool needs_keep = true;
    switch (which) {
        case OUTLETS_BUF_FUSED: src = ctx->cb.r_f; size = 4 * T * d; break;
        case OUTLETS_BUF_NORM_ATTN: src = ctx->cb.a_norm; size = ab * T * d; break;
        case OUTLETS_BUF_Q: src = nullptr; size = ab * T * ctx->qdim; break;
        case OUTLETS_BUF_ATTN: src = ctx->cb.attn; size = ab * T * ctx->qdim; needs_keep = false; break;
        case OUTLETS_BUF_X1: src = ctx->cb.r_x1; size = 4 * T * d; break;
        case OUTLETS_BUF_NORM_MLP: src = ctx->cb.b_norm; size = ab * T * d; break;
        case OUTLETS_BUF_MLP_ACT: src = ctx->cb.mlp; size = ab * T * ctx->F; break;
        case OUTLETS_BUF_X2: src = ctx->cb.r_x2; size = 4 * T * d; break;
        case OUTLETS_BUF_HDRAFT: src = ctx->cb.r_h; size = 4 * T * d; needs_keep = true; break;
        case OUTLETS_BUF_POOLED: src = ctx->cb.pooled; size = 4 * n * 2 * d; needs_keep = false; break;
        case OUTLETS_BUF_NORM_EMB:
            if (!ctx->embed_in) return fail(OUTLETS_ERR_INVALID_ARG, "the context has no input embeddings");
            src = ctx->cb.e_norm; size = ab * T * d; break;
        case OUTLETS_BUF_K_POOL:
        case OUTLETS_BUF_V_POOL:
            src = which == OUTLETS_BUF_K_POOL ? ctx->kpool : ctx->vpool;
            size = ab * static_cast<int64_t>(ctx->cfg.num_pages) * ctx->cfg.n_kv_heads * 16 * ctx->cfg.head_dim;
            needs_keep = false;
            break;
        default: return fail(OUTLETS_ERR_INVALID_ARG, "unknown buffer id");
    }
    *n_bytes = size;
    if (needs_keep && !keep) return fail(OUTLETS_ERR_INVALID_ARG, "buffer needs keep_intermediates");
    if (ctx->last_in_scratch && which != OUTLETS_BUF_K_POOL && which != OUTLETS_BUF_V_POOL)
        return fail(OUTLETS_ERR_INVALID_ARG, "the last predict call ran in the static scratch (no-allocation step)");
    if (!dst || nbytes < size) return fail(OUTLETS_ERR_INVALID_ARG, "destination too small");
    HIP_TRY(hipSetDevice(ctx->device), "hipSetDevice");
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (which == OUTLETS_BUF_Q) {
        // queries live in the first n_q*hd columns of the fused qkv rows
        HIP_TRY(hipMemcpy2DAsync(dst, ab * ctx->qdim, ctx->cb.qkv, ab * ctx->qkv_dim, ab * ctx->qdim, T,
                                 hipMemcpyDeviceToDevice, st), "hipMemcpy2DAsync");
    } else if (size) {
        HIP_TRY(hipMemcpyAsync(dst, src, size, hipMemcpyDeviceToDevice, st), "hipMemcpyAsync");
    }
    return OUTLETS_OK;
}

int outlets_profile_enable_groups(outlets_ctx* ctx, uint32_t groups) {
    if (!ctx) return fail(OUTLETS_ERR_INVALID_ARG, "null context");
    (void)hipSetDevice(ctx->device);
    collect_marks(ctx);
    for (int p = 0; p < 2; ++p)
        for (int i = 0; i < OUTLETS_K_COUNT; ++i) { ctx->prof_ms[p][i] = 0.0; ctx->prof_n[p][i] = 0; }
    ctx->prof_mask = groups & ((1u << OUTLETS_K_COUNT) - 1u);
    ctx->prof_on = ctx->prof_mask != 0;
    return OUTLETS_OK;
}

int outlets_profile_enable(outlets_ctx* ctx, int32_t enable) {
    return outlets_profile_enable_groups(ctx, enable ? (1u << OUTLETS_K_COUNT) - 1u : 0u);
}

int outlets_profile_read(outlets_ctx* ctx, int32_t call, int32_t which, double* total_ms,
                         int64_t* launches) {
    if (!ctx || !total_ms || !launches || which < 0 || which >= OUTLETS_K_COUNT || call < 0 || call > 1)
        return fail(OUTLETS_ERR_INVALID_ARG, "bad argument");
    (void)hipSetDevice(ctx->device);
    collect_marks(ctx);
    *total_ms = ctx->prof_ms[call][which];
    *launches = ctx->prof_n[call][which];
    return OUTLETS_OK;
}

int outlets_varlen_meta(int32_t n_req, const int32_t* lens, int32_t* cu_out, int32_t* pos_out,
                        int32_t* last_out) {
    if (n_req < 0 || (n_req > 0 && !lens)) return fail(OUTLETS_ERR_INVALID_ARG, "bad lengths");
    int rc = varlen_meta(n_req, lens, cu_out, pos_out, last_out);
    return rc ? fail(rc, "lengths must be >= 1 and sum below 2^31") : OUTLETS_OK;
}

int outlets_decode_plan(int32_t n_req, const int32_t* pages, int32_t n_kv, int32_t cus, int32_t* counts,
                        int32_t* work, int64_t work_cap, int32_t* cu_segs, int32_t* lane_off,
                        int64_t lane_cap) {
    if (n_req < 1 || !pages || n_kv < 1 || cus < 1 || !counts) return fail(OUTLETS_ERR_INVALID_ARG, "bad sizes");
    int64_t total = 0;
    for (int i = 0; i < n_req; ++i) {
        if (pages[i] < 1) return fail(OUTLETS_ERR_INVALID_ARG, "page counts must be >= 1");
        total += pages[i];
    }
    if (total > INT32_MAX) return fail(OUTLETS_ERR_INVALID_ARG, "page total exceeds 2^31");
    DecodePlan plan;
    try {
        attn_decode_plan(n_req, pages, n_kv, cus, &plan);
    } catch (const std::bad_alloc&) {
        return fail(OUTLETS_ERR_NOMEM, "host allocation failed");
    }
    counts[0] = static_cast<int32_t>(plan.work.size() / 4);
    counts[1] = plan.n_segs;
    counts[2] = plan.n_lanes;
    if (!work && !cu_segs && !lane_off) return OUTLETS_OK;
    if (!work || !cu_segs || !lane_off) return fail(OUTLETS_ERR_INVALID_ARG, "give all three arrays or none");
    if (work_cap < static_cast<int64_t>(plan.work.size()) || lane_cap < static_cast<int64_t>(plan.lanes.size()))
        return fail(OUTLETS_ERR_INVALID_ARG, "capacity too small");
    std::memcpy(work, plan.work.data(), sizeof(int32_t) * plan.work.size());
    std::memcpy(cu_segs, plan.cu_segs.data(), sizeof(int32_t) * plan.cu_segs.size());
    std::memcpy(lane_off, plan.lanes.data(), sizeof(int32_t) * plan.lanes.size());
    return OUTLETS_OK;
}

struct outlets_pager {
    Pager p;
    outlets_pager(int32_t a, int32_t b, int32_t c, int32_t d) : p(a, b, c, d) {}
};

int outlets_pager_create(int32_t num_pages, int32_t page_size, int32_t max_slots, int32_t max_seq_len,
                         outlets_pager** out) {
    if (!out) return fail(OUTLETS_ERR_INVALID_ARG, "out is null");
    *out = nullptr;
    if (num_pages <= 0 || page_size <= 0 || max_slots <= 0 || max_seq_len <= 0)
        return fail(OUTLETS_ERR_INVALID_ARG, "sizes must be positive");
    try {
        *out = new outlets_pager(num_pages, page_size, max_slots, max_seq_len);
    } catch (const std::bad_alloc&) {
        return fail(OUTLETS_ERR_NOMEM, "host allocation failed");
    }
    return OUTLETS_OK;
}

int outlets_pager_destroy(outlets_pager* p) {
    delete p;
    return OUTLETS_OK;
}

int outlets_pager_prefill(outlets_pager* p, int32_t n, const int32_t* slots, const int32_t* lens) {
    if (!p || n < 0 || (n > 0 && (!slots || !lens))) return fail(OUTLETS_ERR_INVALID_ARG, "bad argument");
    const char* why = "";
    int rc = p->p.prefill(n, slots, lens, nullptr, &why);
    return rc ? fail(rc, why) : OUTLETS_OK;
}

int outlets_pager_step(outlets_pager* p, int32_t n, const int32_t* slots) {
    if (!p || n < 0 || (n > 0 && !slots)) return fail(OUTLETS_ERR_INVALID_ARG, "bad argument");
    const char* why = "";
    int rc = p->p.step(n, slots, nullptr, &why);
    return rc ? fail(rc, why) : OUTLETS_OK;
}

int outlets_pager_release(outlets_pager* p, int32_t n, const int32_t* slots) {
    if (!p || n < 0 || (n > 0 && !slots)) return fail(OUTLETS_ERR_INVALID_ARG, "bad argument");
    const char* why = "";
    int rc = p->p.release(n, slots, &why);
    return rc ? fail(rc, why) : OUTLETS_OK;
}

int outlets_pager_read(outlets_pager* p, int32_t what, int32_t* out, int64_t cap, int64_t* n_out) {
    if (!p || !out || !n_out) return fail(OUTLETS_ERR_INVALID_ARG, "null argument");
    const std::vector<int32_t>* v;
    if (what == OUTLETS_META_PAGE_TABLE) v = &p->p.table();
    else if (what == OUTLETS_META_SEQ_LEN) v = &p->p.seq_lens();
    else return fail(OUTLETS_ERR_INVALID_ARG, "unknown metadata id");
    *n_out = static_cast<int64_t>(v->size());
    if (cap < *n_out) return fail(OUTLETS_ERR_INVALID_ARG, "output capacity too small");
    std::memcpy(out, v->data(), sizeof(int32_t) * v->size());
    return OUTLETS_OK;
}


// ---------------------------------------------------------------- control plane

struct outlets_sched {
    ControlPlane cp;
    outlets_sched(const SchedPolicy& p, int32_t cap) : cp(p, cap) {}
};

namespace {

int check_policy(int32_t k, int32_t s, int32_t routing, int32_t order) {
    if (k <= 0 || s <= 0) return fail(OUTLETS_ERR_INVALID_ARG, "instances and max_running must be positive");
    if ((routing != OUTLETS_ROUTE_RR && routing != OUTLETS_ROUTE_LB) ||
        (order != OUTLETS_QUEUE_FCFS && order != OUTLETS_QUEUE_SJF))
        return fail(OUTLETS_ERR_INVALID_ARG, "unknown routing or queue order");
    return OUTLETS_OK;
}

}  // namespace

int outlets_pred_tokens(int32_t n, const float* z_hat, int32_t* tokens_out) {
    if (n < 0 || (n > 0 && (!z_hat || !tokens_out))) return fail(OUTLETS_ERR_INVALID_ARG, "bad arguments");
    for (int32_t i = 0; i < n; ++i) tokens_out[i] = pred_tokens_from_z(z_hat[i]);
    return OUTLETS_OK;
}

int outlets_sched_create(int32_t n_instances, int32_t max_running, int32_t routing, int32_t queue_order,
                         int32_t max_requests, outlets_sched** out) {
    if (!out) return fail(OUTLETS_ERR_INVALID_ARG, "out is null");
    *out = nullptr;
    int rc = check_policy(n_instances, max_running, routing, queue_order);
    if (rc) return rc;
    if (max_requests <= 0) return fail(OUTLETS_ERR_INVALID_ARG, "max_requests must be positive");
    SchedPolicy p;
    p.instances = n_instances;
    p.max_running = max_running;
    p.routing = routing;
    p.order = queue_order;
    try {
        *out = new outlets_sched(p, max_requests);
    } catch (const std::bad_alloc&) {
        return fail(OUTLETS_ERR_NOMEM, "host allocation failed");
    }
    return OUTLETS_OK;
}

int outlets_sched_destroy(outlets_sched* s) {
    delete s;
    return OUTLETS_OK;
}

int outlets_sched_submit(outlets_sched* s, int32_t n, const int32_t* ids, const int32_t* pred_tokens,
                         int32_t* instance_out) {
    if (!s || n < 0 || (n > 0 && (!ids || !pred_tokens || !instance_out)))
        return fail(OUTLETS_ERR_INVALID_ARG, "bad arguments");
    const char* why = "";
    int rc = s->cp.check_submit(n, ids, pred_tokens, &why);
    if (rc) return fail(rc, why);
    for (int32_t i = 0; i < n; ++i) instance_out[i] = s->cp.submit(ids[i], pred_tokens[i]);
    return OUTLETS_OK;
}

int outlets_sched_admit(outlets_sched* s, int32_t instance, int32_t cap, int32_t* ids_out, int32_t* n_out) {
    if (!s || !n_out || cap < 0 || (cap > 0 && !ids_out)) return fail(OUTLETS_ERR_INVALID_ARG, "bad arguments");
    if (instance < 0 || instance >= s->cp.instances()) return fail(OUTLETS_ERR_INVALID_ARG, "instance out of range");
    *n_out = s->cp.admit(instance, cap, ids_out);
    return OUTLETS_OK;
}

int outlets_sched_iteration(outlets_sched* s, int32_t instance) {
    if (!s) return fail(OUTLETS_ERR_INVALID_ARG, "null control plane");
    if (instance < 0 || instance >= s->cp.instances()) return fail(OUTLETS_ERR_INVALID_ARG, "instance out of range");
    s->cp.iteration(instance);
    return OUTLETS_OK;
}

int outlets_sched_finish(outlets_sched* s, int32_t n, const int32_t* ids) {
    if (!s || n < 0 || (n > 0 && !ids)) return fail(OUTLETS_ERR_INVALID_ARG, "bad arguments");
    std::vector<char> seen(static_cast<size_t>(s->cp.capacity()), 0);
    for (int32_t i = 0; i < n; ++i) {
        if (ids[i] < 0 || ids[i] >= s->cp.capacity()) return fail(OUTLETS_ERR_INVALID_ARG, "request id out of range");
        if (!s->cp.is_running(ids[i])) return fail(OUTLETS_ERR_INVALID_ARG, "request is not running");
        if (seen[ids[i]]) return fail(OUTLETS_ERR_INVALID_ARG, "repeated request id");
        seen[ids[i]] = 1;
    }
    for (int32_t i = 0; i < n; ++i) s->cp.finish(ids[i]);
    return OUTLETS_OK;
}

int outlets_sched_read(outlets_sched* s, int32_t instance, int64_t* load, int32_t* n_waiting,
                       int32_t* n_running) {
    if (!s) return fail(OUTLETS_ERR_INVALID_ARG, "null control plane");
    if (instance < 0 || instance >= s->cp.instances()) return fail(OUTLETS_ERR_INVALID_ARG, "instance out of range");
    if (load) *load = s->cp.load(instance);
    if (n_waiting) *n_waiting = s->cp.n_waiting(instance);
    if (n_running) *n_running = static_cast<int32_t>(s->cp.running(instance).size());
    return OUTLETS_OK;
}

int outlets_sched_simulate(const outlets_sim_config* cfg, int32_t n, const int64_t* arrival_us,
                           const int32_t* out_len, const int32_t* pred_tokens, int32_t* instance_out,
                           int64_t* start_us_out, int64_t* finish_us_out) {
    if (!cfg || n < 0) return fail(OUTLETS_ERR_INVALID_ARG, "bad arguments");
    int rc = check_policy(cfg->n_instances, cfg->max_running, cfg->routing, cfg->queue_order);
    if (rc) return rc;
    if (cfg->iter_base_us < 0 || cfg->iter_per_seq_us < 0)
        return fail(OUTLETS_ERR_INVALID_ARG, "iteration times must be >= 0");
    if (n == 0) return OUTLETS_OK;
    if (!arrival_us || !out_len || !pred_tokens || !instance_out || !start_us_out || !finish_us_out)
        return fail(OUTLETS_ERR_INVALID_ARG, "null array");
    if (arrival_us[0] < 0) return fail(OUTLETS_ERR_INVALID_ARG, "arrival times must be >= 0");
    SimConfig sc;
    sc.policy.instances = cfg->n_instances;
    sc.policy.max_running = cfg->max_running;
    sc.policy.routing = cfg->routing;
    sc.policy.order = cfg->queue_order;
    sc.iter_base_us = cfg->iter_base_us;
    sc.iter_per_seq_us = cfg->iter_per_seq_us;
    const char* why = "";
    try {
        rc = simulate(sc, n, arrival_us, out_len, pred_tokens, instance_out, start_us_out, finish_us_out, &why);
    } catch (const std::bad_alloc&) {
        return fail(OUTLETS_ERR_NOMEM, "host allocation failed");
    }
    return rc ? fail(rc, why) : OUTLETS_OK;
}

int outlets_sched_metrics(int32_t n, const int64_t* arrival_us, const int32_t* out_len,
                          const int64_t* finish_us, int32_t short_below, int32_t long_from,
                          double* out) {
    if (n < 0 || !out || (n > 0 && (!arrival_us || !out_len || !finish_us)))
        return fail(OUTLETS_ERR_INVALID_ARG, "bad arguments");
    const double nan = std::nan("");
    for (int i = 0; i < 6; ++i) out[i] = nan;
    if (n == 0) return OUTLETS_OK;
    std::vector<double> cls[3];
    double lat_sum = 0.0;
    int64_t tokens = 0, t0 = arrival_us[0], t1 = finish_us[0];
    for (int32_t i = 0; i < n; ++i) {
        const double lat = static_cast<double>(finish_us[i] - arrival_us[i]) / 1e6;
        lat_sum += lat;
        tokens += out_len[i];
        t0 = std::min(t0, arrival_us[i]);
        t1 = std::max(t1, finish_us[i]);
        cls[out_len[i] < short_below ? 0 : (out_len[i] < long_from ? 1 : 2)].push_back(lat);
    }
    const double span = static_cast<double>(t1 - t0) / 1e6;
    out[0] = span > 0 ? static_cast<double>(tokens) / span : INFINITY;
    out[1] = lat_sum / n;
    for (int c = 0; c < 3; ++c) {
        std::vector<double>& v = cls[c];
        if (v.empty()) continue;
        std::sort(v.begin(), v.end());
        const size_t m = v.size();
        out[2 + c] = v[(99 * m + 99) / 100 - 1];
    }
    out[5] = span;
    return OUTLETS_OK;
}

}  // extern "C"
