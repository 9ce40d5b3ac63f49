/*
 * outlets.h -- C ABI of the MI355X (gfx950) OUTLETS length-prediction path.
 *
 * OUTLETS ("Output-Length Prediction from Speculative Decoding Backbones")
 * predicts the remaining output length of LLM requests from an EAGLE-3-style
 * speculative draft backbone:
 *
 *   f_ctx   = W_proj Concat(h_low, h_mid, h_high)              (Eq. 1)
 *   h_draft = one Llama-style draft decoder layer over f_ctx    (Section 4.1)
 *   z_hat   = MLP_len(pooled h_draft) ~ log(1 + remaining len)  (Section 4.2)
 *
 * Static prediction runs once after the prompt (Section 3.2, t = 0:
 * outlets_predict_prefill); dynamic prediction re-predicts after every
 * generated token (Section 3.2, t >= 1: outlets_predict_step) using a paged
 * draft KV cache the library owns.
 *
 * Layer details the paper leaves open, fixed here and in the fp64 oracle:
 *   - pre-norm layer, residual stream starting at f_ctx, RMSNorm eps from the
 *     config, bias-free linears, SwiGLU MLP, final RMSNorm -> h_draft;
 *   - rotate-half RoPE: channel pair (c, c + hd/2) rotated by
 *     p * theta^(-2c/hd), no frequency rescaling;
 *   - plain grouped-query attention (query head h reads KV head
 *     h / (n_q / n_kv)), causal within a request; the attention output gate
 *     (Gated Attention) and the input-embedding concat are optional, off
 *     unless their weights are given;
 *   - head input p = [mean of h_draft over the request's tokens so far ;
 *     h_draft of the newest token], then Linear(2d, H1) + ReLU +
 *     Linear(H1, 1), both with biases.
 *
 * All functions are thread-compatible (one context per thread at a time) and
 * return an int status: OUTLETS_OK (0) or a negative OUTLETS_ERR_* code.
 * No C++ exception crosses this boundary.  outlets_last_error() gives a
 * message for the calling thread's last failure.
 *
 * Memory ownership: the caller owns every buffer passed in (weights,
 * activations, outputs); weights registered by outlets_create must stay
 * valid and unchanged until outlets_destroy.  The library owns the KV page
 * pool, per-slot state (cached length, page list, running pool sum) and its
 * workspace.  Host arrays are read before a call returns.  Device work is
 * queued on the given HIP stream (NULL = the default stream); outputs are
 * valid once the caller synchronises that stream.  All calls on one
 * context must be ordered on one stream (or externally synchronised).
 */
#ifndef OUTLETS_H
#define OUTLETS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------ status codes */
enum {
    OUTLETS_OK = 0,
    OUTLETS_ERR_INVALID_ARG = -1,   /* bad size, pointer, slot, length */
    OUTLETS_ERR_SLOT_BUSY = -2,     /* prefill on a slot that is active */
    OUTLETS_ERR_SLOT_EMPTY = -3,    /* step on a slot that is not active */
    OUTLETS_ERR_OUT_OF_PAGES = -4,  /* KV page pool exhausted */
    OUTLETS_ERR_UNSUPPORTED = -5,   /* format/shape the kernels do not handle */
    OUTLETS_ERR_HIP = -6,           /* HIP runtime error (message has details) */
    OUTLETS_ERR_NOMEM = -7          /* device or host allocation failed */
};

/* ------------------------------------------------------------ formats */
enum {
    OUTLETS_FMT_F32 = 0,    /* IEEE binary32 */
    OUTLETS_FMT_BF16 = 1,   /* bfloat16 (upper half of binary32) */
    OUTLETS_FMT_E4M3 = 2    /* OCP FP8 E4M3 codes + one bf16 scale per output row */
};

/*
 * Model and capacity description.
 *   d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim: draft layer shape;
 *     n_q_heads * head_dim need not equal d_model; n_q_heads must be a
 *     multiple of n_kv_heads; head_dim is 64 or 128.
 *   head_hidden: H1, the length head's hidden width.
 *   rope_theta, rms_eps: RoPE base and RMSNorm epsilon.
 *   weight_fmt: F32 (then act_fmt must be F32), BF16 or E4M3 (act BF16).
 *     With E4M3 only the eight big linears (proj, q, k, v, o, gate, up, down)
 *     are fp8; gains and the head are bf16.  BF16/E4M3 shapes need d_model,
 *     n_q_heads*head_dim, n_kv_heads*head_dim and head_hidden to be
 *     multiples of 256 and ffn_dim a multiple of 128 (the MFMA tiles);
 *     outlets_create returns UNSUPPORTED otherwise.
 *   act_fmt: format of h_low/h_mid/h_high, of h_draft output and of the KV
 *     cache: F32 or BF16.
 *   page_size: tokens per KV page; must be 16.
 *   max_slots: number of request slots (per-request state entries).
 *   max_seq_len: longest request (prompt + generated tokens).
 *   num_pages: KV pages in the pool (each holds page_size tokens of K and V
 *     for every KV head).
 *   max_batch_tokens: largest packed token count one prefill call may pass.
 *   max_batch_requests: largest n_req of one prefill or step call.
 *   keep_intermediates: nonzero keeps every intermediate activation of the
 *     last call in its own buffer so outlets_get_buffer can return it (more
 *     device memory; for testing).
 */
typedef struct outlets_config {
    int32_t d_model;
    int32_t n_q_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t ffn_dim;
    int32_t head_hidden;
    double rope_theta;
    float rms_eps;
    int32_t weight_fmt;
    int32_t act_fmt;
    int32_t page_size;
    int32_t max_slots;
    int32_t max_seq_len;
    int32_t num_pages;
    int32_t max_batch_tokens;
    int32_t max_batch_requests;
    int32_t keep_intermediates;
    int32_t vocab;        /* draft model head vocabulary V (Eq. 2); 0 = no draft head */
} outlets_config;

/*
 * Device pointers to the weights, PyTorch [out, in] row-major layout.
 *   w_proj [d, 3d]  (columns: h_low, h_mid, h_high; Eq. 1)
 *   w_q [n_q*hd, d], w_k [n_kv*hd, d], w_v [n_kv*hd, d], w_o [d, n_q*hd]
 *   w_gate [F, d], w_up [F, d], w_down [d, F]
 *   s_*: bf16 [out] row scales, required for E4M3 and ignored otherwise
 *        (the weight value is decode(code) * scale[row]).
 *   gamma_attn, gamma_mlp, gamma_final [d]: RMSNorm gains
 *   head_w1 [H1, 2d], head_b1 [H1], head_w2 [H1], head_b2 [1]
 *   w_attn_gate [n_q*hd, d] (optional, NULL = plain attention): Gated
 *     Attention (Section 4.1, citing its source for the formula): the
 *     attention output of query head h, channel c is multiplied by
 *     sigmoid((a W_attn_gate^T)[h*hd + c]), a the normed layer input that
 *     also feeds Q/K/V, before W_o.  Stored like the other big linears
 *     (weight_fmt, with s_attn_gate row scales for E4M3).
 *   probe_w1 [H1, 2d], probe_b1 [H1], probe_w2 [H1], probe_b2 [1]
 *     (optional, all or none; small-weight format like head_*): the MLP-probe
 *     baseline (Section 5.1 baselines: an MLP regressor on the frozen target
 *     model's hidden states), see outlets_probe_prefill.
 *   w_lm [V, d] (optional, NULL = no draft head; needs cfg.vocab = V > 0;
 *     weight_fmt, with s_lm row scales for E4M3): the draft model head of
 *     Eq. 2, see outlets_draft_distribution.
 *   embed [V, d] (act_fmt) and gamma_emb [d] (optional, both or none; need
 *     cfg.vocab = V > 0): EAGLE-3 input embeddings, the backbone component
 *     of the Section 5 ablation.  The attention block then reads the 2d-wide
 *     row x = [RMSNorm(embed[token]) * gamma_emb ; RMSNorm(f_ctx) *
 *     gamma_attn]: w_q, w_k, w_v (and w_attn_gate) become [out, 2d] with
 *     the embedding columns first; the residual stream still starts at
 *     f_ctx.  The predict calls then take one token id per row.
 * cfg.vocab > 0 needs w_lm or embed (or both).
 * Element format: weight_fmt for the big linears; F32 for the rest when
 * weight_fmt is F32, BF16 otherwise.
 */
typedef struct outlets_weights {
    const void* w_proj;  const void* s_proj;
    const void* w_q;     const void* s_q;
    const void* w_k;     const void* s_k;
    const void* w_v;     const void* s_v;
    const void* w_o;     const void* s_o;
    const void* w_gate;  const void* s_gate;
    const void* w_up;    const void* s_up;
    const void* w_down;  const void* s_down;
    const void* gamma_attn;
    const void* gamma_mlp;
    const void* gamma_final;
    const void* head_w1;
    const void* head_b1;
    const void* head_w2;
    const void* head_b2;
    const void* w_attn_gate;  const void* s_attn_gate;
    const void* probe_w1;
    const void* probe_b1;
    const void* probe_w2;
    const void* probe_b2;
    const void* w_lm;    const void* s_lm;
    const void* embed;
    const void* gamma_emb;
} outlets_weights;

typedef struct outlets_ctx outlets_ctx;
typedef struct outlets_pager outlets_pager;

/*
 * Create a context on HIP device `device`: validates the config, records the
 * weight pointers (not copied), builds the RoPE cos/sin table on the host in
 * float64 and uploads it as float32, and allocates the KV page pool, the
 * per-slot state and the workspace.  Synchronous.  On failure *out is NULL.
 */
int outlets_create(const outlets_config* cfg, const outlets_weights* weights,
                   int32_t device, outlets_ctx** out);

/* Free everything the context owns.  Synchronises the device first.  NULL is a no-op. */
int outlets_destroy(outlets_ctx* ctx);

/*
 * Static prediction (Section 3.2, t = 0) for n_req new requests.
 *   slots [n_req] (host): slot id of each request, all inactive and distinct.
 *   lens [n_req] (host): prompt length n_i >= 1 of each request.
 *   h_low, h_mid, h_high (device, act_fmt): the target model's hidden states
 *     at the three selected depths (Section 4.1: layers 2, N/2, N-2), packed
 *     varlen in `slots` order: request i owns rows [cu_i, cu_{i+1}) with
 *     cu_0 = 0, cu_{i+1} = cu_i + lens[i]; row r starts at element
 *     r * row_stride (row_stride >= d_model).  One [T, 3d] tensor may be
 *     passed as base, base + d, base + 2d with row_stride 3d.
 *   tokens (device, int32 [T], packed like the states; ignored unless the
 *     context has input embeddings, then required): the token id paired
 *     with each row (in EAGLE-3 the token that follows the row's position;
 *     the caller decides the pairing).  An id outside [0, V) cannot be
 *     reported from the device: its embedding row is taken as zero.
 *   z_out (device, float32 [n_req]): z_hat_i, the predicted log(1 + L_i).
 *   hdraft_out (device, act_fmt [T, d] or NULL): h_draft of every token.
 *   stream: hipStream_t (NULL = default stream).
 * Prompt tokens take positions 0..n_i-1.  Each slot receives ceil(n_i/16)
 * pages: lowest free page ids first, requests in argument order.  All checks
 * and the page allocation happen before any device work; on any error the
 * state is unchanged.  Check order: n_req range and pointers, then per
 * request slot range / repetition / length, then busy slots, then page
 * availability.  n_req == 0 is a no-op.
 */
int outlets_predict_prefill(outlets_ctx* ctx, int32_t n_req, const int32_t* slots,
                            const int32_t* lens, const void* h_low, const void* h_mid,
                            const void* h_high, int64_t row_stride, const int32_t* tokens,
                            float* z_out, void* hdraft_out, void* stream);

/*
 * Dynamic prediction (Section 3.2, t >= 1): one generated token per request.
 *   slots [n_req] (host): active, distinct slots.
 *   h_low, h_mid, h_high (device, act_fmt [n_req rows], row_stride): states
 *     of the newly generated token y_t, row i for slots[i].
 *   tokens (device int32 [n_req]; as in outlets_predict_prefill).
 *   z_out (device float32 [n_req]): z_hat_t, the predicted log(1 + r_t).
 *   hdraft_out (device act_fmt [n_req, d] or NULL).
 * The token takes position (cached length) and attends over every cached key
 * plus itself; the running mean in the head input covers prompt and
 * generated tokens.  A slot takes a new page exactly when its cached length
 * is a multiple of 16 before the append.  Check order: n_req range and
 * pointers, slot range / repetition, inactive slots, full slots
 * (cached length == max_seq_len), page availability; on error the state is
 * unchanged.
 */
int outlets_predict_step(outlets_ctx* ctx, int32_t n_req, const int32_t* slots,
                         const void* h_low, const void* h_mid, const void* h_high,
                         int64_t row_stride, const int32_t* tokens, float* z_out,
                         void* hdraft_out, void* stream);

/*
 * outlets_predict_step without device allocation, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Arguments, results, state changes and
 * error codes are those of outlets_predict_step (same kernels and split
 * plans, so the same bits), except:
 *   - the call's per-call device buffers (activations, split-K / split-KV /
 *     head partial sums, token metadata) live in the library's static
 *     scratch array of 256 MiB on each device, not in the context: a step
 *     whose buffers exceed it fails with OUTLETS_ERR_INVALID_ARG and no
 *     state change (8B shape: up to 512 requests fit);
 *   - every no-allocation call on one device shares that array and it keeps
 *     the last call's contents: calls that overlap on one device (several
 *     contexts, streams or threads) race;
 *   - contexts created with keep_intermediates are refused
 *     (OUTLETS_ERR_UNSUPPORTED); after this call outlets_get_buffer (other
 *     than the KV pools), the device entries of outlets_get_meta and
 *     outlets_draft_distribution fail with OUTLETS_ERR_INVALID_ARG until the
 *     next outlets_predict_prefill / outlets_predict_step;
 *   - per-kernel timing (outlets_profile_enable) records nothing for it.
 * It calls no hipMalloc / hipFree; nothing in the scratch needs clearing
 * (every kernel writes what a later one reads).
 */
int outlets_predict_step_noalloc(outlets_ctx* ctx, int32_t n_req, const int32_t* slots,
                                 const void* h_low, const void* h_mid, const void* h_high,
                                 int64_t row_stride, const int32_t* tokens, float* z_out,
                                 void* hdraft_out, void* stream);

/* End requests: frees their pages and state.  Inactive slots are a no-op;
 * an out-of-range or repeated slot fails with no change. */
int outlets_release(outlets_ctx* ctx, int32_t n, const int32_t* slots);

/*
 * MLP-probe baseline (the comparison predictor of Section 5.1: an MLP on
 * the target model's hidden states, no draft layer).  The probe reads one
 * target-state tensor `h` (e.g. the mid-depth state) and runs the length
 * head's pooling and MLP on it with the probe weights:
 *   z_i = probe_w2 . relu(probe_w1 [mean of h over the tokens so far ;
 *         h of the newest token] + probe_b1) + probe_b2.
 * Probe slots are independent of the draft path's slots (same id range).
 * Requires probe weights at create (else OUTLETS_ERR_UNSUPPORTED).
 *
 * outlets_probe_prefill: static probe prediction for n_req new requests;
 *   h (device, act_fmt) packed like outlets_predict_prefill's states, row r at
 *   element r * row_stride; z_out [n_req] device fp32.  Errors (state
 *   unchanged): bad n_req / pointers / slot ids / repeats (INVALID_ARG),
 *   an active probe slot (SLOT_BUSY), len < 1 or sum(lens) >
 *   max_batch_tokens (INVALID_ARG).
 * outlets_probe_step: one new token's state per active probe slot (row i of
 *   h); updates the slot's running sum.  Inactive slot: SLOT_EMPTY.
 * outlets_probe_release: ends probe slots (inactive ones are a no-op).
 */
int outlets_probe_prefill(outlets_ctx* ctx, int32_t n_req, const int32_t* slots, const int32_t* lens,
                          const void* h, int64_t row_stride, float* z_out, void* stream);
int outlets_probe_step(outlets_ctx* ctx, int32_t n_req, const int32_t* slots, const void* h,
                       int64_t row_stride, float* z_out, void* stream);
int outlets_probe_release(outlets_ctx* ctx, int32_t n, const int32_t* slots);

/*
 * Draft model head (Eq. 2): for each request of the last outlets_predict_*
 * call, P_draft(y_{t+1} | y_{1:t}) = softmax(W_lm h_t^draft) over the V
 * vocabulary entries, h_t^draft the draft state of the request's newest
 * token (the same state the length head reads).
 *   n_req: must equal the last predict call's request count.
 *   p_out (device): fp32 [n_req, V] row-major probabilities.
 * Must be queued before the next predict or probe call on the context (it
 * reads that call's pooled draft states).  Errors: no draft head, w_lm
 * NULL (UNSUPPORTED), n_req mismatch or null p_out (INVALID_ARG).
 */
int outlets_draft_distribution(outlets_ctx* ctx, int32_t n_req, float* p_out, void* stream);

/* ------------------------------------------------------------ inspection */
enum {
    OUTLETS_META_PAGE_TABLE = 0,        /* host table [max_slots, max_pages_per_seq], -1 = none */
    OUTLETS_META_SEQ_LEN = 1,           /* host cached length per slot [max_slots] */
    OUTLETS_META_DEV_PAGE_TABLE = 2,    /* the device copy the kernels read */
    OUTLETS_META_DEV_CU_SEQLENS = 3,    /* last call, device: [n_req + 1] token offsets */
    OUTLETS_META_DEV_POSITIONS = 4,     /* last call, device: [T] token positions */
    OUTLETS_META_DEV_LAST_IDX = 5,      /* last call, device: [n_req] row of the newest token */
    OUTLETS_META_DEV_TOKEN_SLOT = 6     /* last call, device: [T] slot of each token */
};

/*
 * Copy integer metadata into host memory `out` (capacity `cap` int32s);
 * *n_out receives the element count.  Device entries synchronise the device.
 * Fails with INVALID_ARG if cap is too small.
 */
int outlets_get_meta(outlets_ctx* ctx, int32_t what, int32_t* out, int64_t cap, int64_t* n_out);

enum {
    OUTLETS_BUF_FUSED = 0,      /* f_ctx, float32 [T, d] */
    OUTLETS_BUF_NORM_ATTN = 1,  /* RMSNorm(f_ctx), act [T, d] */
    OUTLETS_BUF_Q = 2,          /* queries after RoPE, act [T, n_q*hd] */
    OUTLETS_BUF_ATTN = 3,       /* attention output, act [T, n_q*hd] */
    OUTLETS_BUF_X1 = 4,         /* f + attn W_o^T, float32 [T, d] */
    OUTLETS_BUF_NORM_MLP = 5,   /* RMSNorm(x1), act [T, d] */
    OUTLETS_BUF_MLP_ACT = 6,    /* silu(gate) * up, act [T, F] */
    OUTLETS_BUF_X2 = 7,         /* x1 + mlp, float32 [T, d] */
    OUTLETS_BUF_HDRAFT = 8,     /* h_draft, float32 [T, d] */
    OUTLETS_BUF_POOLED = 9,     /* head input p, float32 [n_req, 2d] */
    OUTLETS_BUF_K_POOL = 10,    /* key pages, act [num_pages, n_kv, 16, hd] */
    OUTLETS_BUF_V_POOL = 11,    /* value pages, transposed: act [num_pages, n_kv, hd, 16] */
    OUTLETS_BUF_NORM_EMB = 12   /* RMSNorm(embed[token]) * gamma_emb, act [T, d] (input embeddings) */
};

/*
 * Copy an activation of the last call (rows of that call only) or a KV pool
 * into caller device memory `dst` (`nbytes` capacity) on `stream`;
 * *n_bytes receives the size.  Buffers 0..2, 4..8 and 12 need
 * keep_intermediates (ATTN, POOLED and the pools are always kept; h_draft of
 * every row is otherwise available through the predict calls' hdraft_out);
 * NORM_EMB needs input embeddings.
 */
int outlets_get_buffer(outlets_ctx* ctx, int32_t which, void* dst, int64_t nbytes,
                       int64_t* n_bytes, void* stream);

/* ------------------------------------------------------------ per-kernel timing */
enum {
    OUTLETS_K_META = 0,         /* page-table scatter + token metadata */
    OUTLETS_K_FUSE_GEMM = 1,    /* Eq. 1 projection */
    OUTLETS_K_NORM = 2,         /* the RMSNorms (and the embedding gather + norm) */
    OUTLETS_K_QKV_GEMM = 3,
    OUTLETS_K_ROPE_KV = 4,      /* rotary embedding + paged K/V write */
    OUTLETS_K_ATTN = 5,
    OUTLETS_K_O_GEMM = 6,
    OUTLETS_K_GATE_UP_GEMM = 7, /* gate/up projection with the SwiGLU epilogue */
    OUTLETS_K_DOWN_GEMM = 8,
    OUTLETS_K_POOL = 9,         /* pooling (in prefill calls with the final RMSNorm, fused) */
    OUTLETS_K_HEAD = 10,        /* length head (both layers) */
    OUTLETS_K_COUNT = 11
};

/*
 * enable != 0 starts recording a HIP event pair around every kernel launch
 * of later calls (on the call's stream) and clears the totals; 0 stops.
 * Timing adds a little launch overhead; leave it off in production.
 */
int outlets_profile_enable(outlets_ctx* ctx, int32_t enable);

/*
 * Like outlets_profile_enable, but records event pairs only around the
 * kernel groups whose bit is set in `groups` (bit k = group OUTLETS_K_k;
 * bits at or above OUTLETS_K_COUNT are ignored); 0 stops.  Timing one group
 * (e.g. the dominant kernel) perturbs the calls far less than timing all of
 * them.  Clears the totals.
 */
int outlets_profile_enable_groups(outlets_ctx* ctx, uint32_t groups);

/*
 * Total milliseconds and launch count recorded for kernel group `which`
 * (OUTLETS_K_*) inside prefill calls (call = 0) or step calls (call = 1)
 * since profiling was enabled.  Synchronises on the recorded events.
 */
int outlets_profile_read(outlets_ctx* ctx, int32_t call, int32_t which, double* total_ms,
                         int64_t* launches);

/* Message for the calling thread's last failed call ("" if none). */
const char* outlets_last_error(void);

/* ------------------------------------------------------------ host-only entry points
 * These run on the CPU and touch no GPU; the context uses the same code. */

/*
 * Varlen metadata of packed prompts (host arrays): cu_out [n_req + 1]
 * (exclusive prefix sum, cu_out[0] = 0), pos_out [T] (0..n_i-1 per request)
 * and last_out [n_req] (cu_{i+1} - 1).  Any output may be NULL.  Lengths
 * must be >= 1.
 */
int outlets_varlen_meta(int32_t n_req, const int32_t* lens, int32_t* cu_out,
                        int32_t* pos_out, int32_t* last_out);

/*
 * The split-KV work plan that outlets_predict_step uses for decode attention
 * (bf16, head dim 128; Section 3.2 dynamic prediction reads the whole paged
 * cache of every request at each step).  pages[i] = pages of request i's
 * cache including the step's token (>= 1); n_kv = KV heads; cus = compute
 * units.  The pages, requests in order, are cut into n_lanes contiguous
 * ranges whose lengths differ by at most one page (one wave per range and
 * KV head); a range's part in one request is a segment (one partial softmax
 * record), walked in pieces of at most 64 pages.  Outputs (host):
 *   counts[3] = n_pieces, n_segs, n_lanes (always written);
 *   work [4 n_pieces] = (request, first page, end page, segment) per piece;
 *   cu_segs [n_req + 1] = first segment of each request (segments of a
 *   request are consecutive, in page order);
 *   lane_off [n_lanes + 1] = first piece of each range.
 * work, cu_segs and lane_off may all be NULL (counts only); otherwise all
 * three are written, and capacities below 4 n_pieces (work_cap) or
 * n_lanes + 1 (lane_cap) fail with OUTLETS_ERR_INVALID_ARG and write only
 * counts.  Bad sizes or a page count below 1 fail with INVALID_ARG.
 */
int outlets_decode_plan(int32_t n_req, const int32_t* pages, int32_t n_kv, int32_t cus, int32_t* counts,
                        int32_t* work, int64_t work_cap, int32_t* cu_segs, int32_t* lane_off,
                        int64_t lane_cap);

/* A stand-alone instance of the context's page allocator (host memory only). */
int outlets_pager_create(int32_t num_pages, int32_t page_size, int32_t max_slots,
                         int32_t max_seq_len, outlets_pager** out);
int outlets_pager_destroy(outlets_pager* p);
int outlets_pager_prefill(outlets_pager* p, int32_t n, const int32_t* slots, const int32_t* lens);
int outlets_pager_step(outlets_pager* p, int32_t n, const int32_t* slots);
int outlets_pager_release(outlets_pager* p, int32_t n, const int32_t* slots);
/* what: OUTLETS_META_PAGE_TABLE or OUTLETS_META_SEQ_LEN. */
int outlets_pager_read(outlets_pager* p, int32_t what, int32_t* out, int64_t cap, int64_t* n_out);

/* ------------------------------------------------------------ control plane
 * The consumer of the static prediction r_hat_0 in disaggregated serving
 * (Section 5, system-level evaluation): routing of arriving requests over K
 * decode instances and the admission order of each instance's queue.  Host
 * code only (no GPU), thread-compatible.
 *   routing OUTLETS_ROUTE_RR: the i-th submitted request goes to instance
 *     i mod K.  OUTLETS_ROUTE_LB: to the instance with the lowest estimated
 *     remaining work, the sum of predicted remaining lengths of its waiting
 *     (pred) and running (max(pred - generated, 0)) requests; ties go to the
 *     lowest instance index.
 *   queue OUTLETS_QUEUE_FCFS: admission in submission order.
 *     OUTLETS_QUEUE_SJF: shortest predicted length first, ties in
 *     submission order.  Admission is non-preemptive.
 * Predicted lengths are whole tokens (outlets_pred_tokens converts the
 * length head's z_hat).
 */
enum { OUTLETS_ROUTE_RR = 0, OUTLETS_ROUTE_LB = 1 };
enum { OUTLETS_QUEUE_FCFS = 0, OUTLETS_QUEUE_SJF = 1 };

typedef struct outlets_sched outlets_sched;

/*
 * z_hat (host float [n], the length head's log(1 + length) estimates) ->
 * tokens_out (host int32 [n]): floor(max(0, expm1(z)) + 0.5), NaN -> 0,
 * capped at 2^31 - 1.
 */
int outlets_pred_tokens(int32_t n, const float* z_hat, int32_t* tokens_out);

/*
 * An online control plane for K = n_instances decode instances running at
 * most max_running requests each; request ids are the caller's, in
 * [0, max_requests), and may be reused once finished.
 */
int outlets_sched_create(int32_t n_instances, int32_t max_running, int32_t routing,
                         int32_t queue_order, int32_t max_requests, outlets_sched** out);
int outlets_sched_destroy(outlets_sched* s);

/*
 * Route n arriving requests in argument order; instance_out [n] receives
 * each one's instance, and each joins that instance's queue.  All checks
 * come first (ids in range and idle, no repeats, pred_tokens >= 0: else
 * INVALID_ARG, or SLOT_BUSY for an id still waiting or running) and a failed
 * call changes nothing.
 */
int outlets_sched_submit(outlets_sched* s, int32_t n, const int32_t* ids, const int32_t* pred_tokens,
                         int32_t* instance_out);

/*
 * Admit up to min(cap, max_running - running) waiting requests of
 * `instance` in queue order: ids_out [cap] receives them, *n_out the count.
 * Call it when the instance starts a decode iteration.
 */
int outlets_sched_admit(outlets_sched* s, int32_t instance, int32_t cap, int32_t* ids_out, int32_t* n_out);

/* One decode iteration of `instance` finished: each running request there
 * generated one token (its predicted remaining length drops by one while
 * positive). */
int outlets_sched_iteration(outlets_sched* s, int32_t instance);

/* Requests that finished; each must be running (else INVALID_ARG, no change). */
int outlets_sched_finish(outlets_sched* s, int32_t n, const int32_t* ids);

/* Estimated remaining work (predicted tokens), queue length and running
 * count of `instance`; any output may be NULL. */
int outlets_sched_read(outlets_sched* s, int32_t instance, int64_t* load, int32_t* n_waiting,
                       int32_t* n_running);

/*
 * Discrete-event run of the decode cluster (the setting of the paper's
 * saturation experiment: one prefill instance feeding K decode instances)
 * over a request trace, using the control plane above.  Each instance runs
 * continuous-batching iterations back to back while it has running
 * requests; an iteration with b running requests lasts iter_base_us +
 * iter_per_seq_us * b microseconds and gives each one token; waiting
 * requests are admitted only when an iteration starts (or on arrival at an
 * idle instance); a request finishes at the end of the iteration that makes
 * its out_len-th token.  Events at one instant: iteration ends (instance
 * order), then arrivals (trace order), then admissions and iteration starts.
 *   arrival_us [n] (host, >= 0, nondecreasing), out_len [n] (true output
 *   lengths >= 1), pred_tokens [n] (>= 0).
 *   instance_out [n], start_us_out [n] (admission time), finish_us_out [n].
 * Errors: bad config or inputs (INVALID_ARG, nothing written).
 */
typedef struct outlets_sim_config {
    int32_t n_instances;
    int32_t max_running;
    int32_t routing;
    int32_t queue_order;
    int64_t iter_base_us;
    int64_t iter_per_seq_us;
} outlets_sim_config;

int outlets_sched_simulate(const outlets_sim_config* cfg, int32_t n, const int64_t* arrival_us,
                           const int32_t* out_len, const int32_t* pred_tokens, int32_t* instance_out,
                           int64_t* start_us_out, int64_t* finish_us_out);

/*
 * Serving metrics of a run: out [6] = throughput (generated tokens / (last
 * finish - first arrival), tokens/s), mean latency (s), P99 latency (s,
 * nearest rank: the ceil(0.99 m)-th smallest of m) of requests with out_len
 * < short_below, in [short_below, long_from), and >= long_from (NaN for an
 * empty class), and the makespan (s).  Latency = finish - arrival.
 */
int outlets_sched_metrics(int32_t n, const int64_t* arrival_us, const int32_t* out_len,
                          const int64_t* finish_us, int32_t short_below, int32_t long_from,
                          double* out);

#ifdef __cplusplus
}
#endif

#endif /* OUTLETS_H */
