// Launch interface of the gfx950 kernels (library-internal).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>
#include <vector>

namespace outlets {

// ---------------------------------------------------------------- GEMM
// C[M, N] = A[M, K] . B[N, K]^T, fp32 accumulation.
//
// A: activations; the K axis may come from up to three pointers, each
//    supplying `kseg` consecutive columns (the fused projection reads
//    h_low | h_mid | h_high this way without materialising the concat).
// B: weights, [out, in] row-major.  Rows come from up to three pointers
//    (`nend[s]` = exclusive end of block s in logical rows: Wq | Wk | Wv), or,
//    with `paired`, logical rows alternate 32 rows of p[0] and 32 rows of
//    p[1] (gate | up) so one output tile holds matching gate/up columns.
//    E4M3 weights carry one bf16 scale per physical row.
struct GemmA {
    const void* p[3];
    int64_t ld;      // elements between rows
    int32_t kseg;    // columns per pointer (K when one pointer)
};

struct GemmB {
    const void* p[4];            // up to 4 row segments (e.g. Wq | Wk | Wv | W_gate)
    const uint16_t* scale[4];
    int32_t nend[4];             // cumulative row ends; unused entries = N
    int32_t paired;
    int64_t ld;
};

enum Epilogue : int {
    EPI_STORE_F32 = 0,  // C (f32) = acc
    EPI_STORE_ACT = 1,  // C (act format) = acc
    EPI_RESID_F32 = 2,  // C (f32) = resid + acc   (C may alias resid)
    EPI_SWIGLU = 3,     // C (act) [M, N/2] = silu(gate) * up   (requires paired B)
    EPI_PARTIAL = 4,    // C (f32) + split * split_stride = acc over the split's K range
    EPI_PARTIAL_TILE = 5, // internal: per-tile fp32 blocks of the K-split tail of a large GEMM
    EPI_QKV_ROPE = 6    // q|k|v|gate columns (bf16, head dim 128): q rotated and stored to C,
                        // k rotated and v written into their KV pages, gate stored to C
};

// Rotary embedding and paged K/V write of EPI_QKV_ROPE (rows are tokens):
// the layout of launch_rope_kv.
struct RopeKV {
    const int32_t* tok_pos;
    const int32_t* tok_slot;
    const int32_t* page_table;
    int32_t max_pages, n_q, n_kv;
    uint16_t* kpool;
    uint16_t* vpool;
    const float* cos_t;
    const float* sin_t;
};

struct GemmC {
    void* c;
    int64_t ldc;
    const float* resid;
    int64_t ldr;
    int64_t split_stride;
    RopeKV rope;
};

enum Fmt : int { FMT_F32 = 0, FMT_BF16 = 1, FMT_E4M3 = 2 };

// Checks the shape against what the selected kernel handles; returns 0 or an
// OUTLETS_ERR_* code (and a reason).  act_fmt is the format of A and of act
// outputs; w_fmt of B.
int gemm_check(int act_fmt, int w_fmt, int epi, int M, int N, int K, const GemmA& a,
               const GemmB& b, int splits, const char** why);
// `ws` (fp32 scratch of ws_bytes, may be null) enables the small-M split-K
// path (gemm_splitk_plan splits > 1): partial sums, then a fixed-order reduce
// that applies the epilogue.
void gemm_launch(int act_fmt, int w_fmt, int epi, int M, int N, int K, const GemmA& a,
                 const GemmB& b, const GemmC& c, int splits, hipStream_t st,
                 float* ws = nullptr, size_t ws_bytes = 0);
int gemm_splitk_plan(int w_fmt, int epi, int M, int N, int K);
// The partial-sum half of a split-K call: when gemm_launch would split this
// call (epilogue `epi`, workspace ws of ws_bytes), launches only the split
// GEMM, leaving S fp32 planes [M, N] in ws (plane s at ws + s M N), and
// returns S; otherwise launches nothing and returns 0.  A row kernel that
// takes a RowSum then finishes the call (see launch_rmsnorm_sum).
int gemm_launch_partials(int act_fmt, int w_fmt, int epi, int M, int N, int K, const GemmA& a,
                         const GemmB& b, float* ws, size_t ws_bytes, hipStream_t st);
// Bytes of fp32 workspace gemm_launch uses for this call when given ws_bytes
// (0 when it splits nothing); a call given exactly these bytes takes the
// same plan as with ws_bytes.
size_t gemm_workspace_bytes(int w_fmt, int epi, int M, int N, int K, size_t ws_bytes);
int gemm_device_cus();   // compute units of the current device
// Whether gemm_launch takes EPI_QKV_ROPE for this layout (bf16 activations,
// head dim 128; N = q|k|v[|gate] columns); otherwise store with
// EPI_STORE_ACT and run launch_rope_kv.  With a K split the reduce kernel
// applies the same epilogue.
bool gemm_qkv_rope_fusable(int act_fmt, int w_fmt, int n_q, int n_kv, int hd, int N);

// ---------------------------------------------------------------- elementwise / rows
// A call's metadata block from pinned host-coherent memory (`host_meta`,
// `count` int32: req_off[n + 1] | req_slot[n] | req_start[n] | n_pairs
// (index, page) pairs | the rest) into d_meta; applies the pairs to
// page_table and writes tok_slot[T] (slot of each token), tok_pos[T]
// (req_start + index within the request) and last_idx[n] (row of each
// request's newest token).  With n_req = n_pairs = 0 it only copies (the
// other pointers may then be null).  The host must not rewrite host_meta
// until the kernel has run.
void launch_meta_fetch(const int32_t* host_meta, int count, int n_req, int n_pairs, int32_t* d_meta,
                       int32_t* page_table, int32_t* tok_slot, int32_t* tok_pos, int32_t* last_idx, hipStream_t st);

// Row x[r] of a split-K GEMM's output: the S partial planes summed in split
// order, plus resid[r] when resid is set (the fp32 residual the GEMM's
// epilogue would add); stored to out[r] when out is set (it may alias resid).
struct RowSum {
    const float* part;
    int S;
    int64_t plane;   // elements between partial planes (M N)
    int64_t ldp;     // elements between partial rows (N)
    const float* resid;
    int64_t ldr;
    float* out;
    int64_t ldo;
};
// Whether the row kernels take a RowSum for rows of d elements.
bool rowsum_supported(int d);

// y = x / sqrt(mean(x^2) + eps) * gamma per row; x fp32; y in act format
// (either output may be null; y2 is an fp32 copy and may alias x).
void launch_rmsnorm(int act_fmt, int gamma_fmt, int rows, int d, const float* x, int64_t ldx,
                    const void* gamma, float eps, void* y, int64_t ldy, float* y2,
                    int64_t ldy2, hipStream_t st);

// launch_rmsnorm of the rows a RowSum forms (rowsum_supported(d) must hold).
void launch_rmsnorm_sum(int act_fmt, int gamma_fmt, int rows, int d, const RowSum& rs, const void* gamma,
                        float eps, void* y, int64_t ldy, hipStream_t st);

// EAGLE-3 input embeddings: y[r] = RMSNorm(embed[tok[r]]) * gamma for `rows`
// token ids; embed [vocab, d] and y in act format, gamma in gamma_fmt.  Ids
// outside [0, vocab) give zero rows.
void launch_embed_norm(int act_fmt, int gamma_fmt, int rows, int d, int vocab, const int32_t* tok,
                       const void* embed, const void* gamma, float eps, void* y, int64_t ldy,
                       hipStream_t st);

// RoPE on q (in place) and k; k, v scattered into the page pools.
void launch_rope_kv(int act_fmt, int ntok, void* qkv, int64_t ld, const int32_t* tok_slot,
                    const int32_t* tok_pos, const int32_t* page_table, int max_pages,
                    void* kpool, void* vpool, const float* cos_t, const float* sin_t,
                    int n_q, int n_kv, int hd, hipStream_t st);

bool attn_supported(int n_q, int n_kv, int hd);
bool attn_prefill_mfma_supported(int act_fmt, int n_q, int n_kv, int hd);
// Queries per prefill attention work item (a multiple of 32) for a call of
// `tokens` prompt tokens over n_req requests.
int attn_prefill_query_tile(int n_q, int n_kv, int64_t tokens, int n_req);

// Attention kernels: `gate` (nullable) points at the Gated Attention gate
// values of token/request row 0, laid out like q (row stride ldq, query head h
// at h * hd); each output element is multiplied by sigmoid of its gate value.
//
// Causal prefill attention on MFMA (bf16, hd 128).  work[2 * i], work[2 * i + 1]
// = (request, query tile) of workgroup row i; req_off = token offsets.
void launch_attn_prefill(int n_work, const int32_t* work, int qtile, const void* qkv, int64_t ldq, void* out,
                         int64_t ldo, const int32_t* req_off, const int32_t* req_slot,
                         const int32_t* page_table, int max_pages, const void* kpool,
                         const void* vpool, int n_q, int n_kv, const void* gate, hipStream_t st);

// Decode attention (bf16, hd 128, one query per request).  The step's pages,
// requests in order, are cut into n_lanes equal ranges, one per wave and KV
// head; a range's part in one request is a segment (one fp32 partial record
// per segment and query head), walked in pieces of at most 64 pages.
// DecodePlan: work[4 i .. 4 i + 3] = (request, first page, end page, segment)
// of piece i; lanes = n_lanes + 1 piece offsets; cu_segs[n_req + 1] = first
// segment of each request; part = fp32 scratch [n_segs, n_q,
// attn_decode_record_floats()].  Queries are row r of q for request r.
struct DecodePlan {
    std::vector<int32_t> work, cu_segs, lanes;
    int n_lanes = 0, n_segs = 0;
};
void attn_decode_plan(int n_req, const int32_t* pages, int n_kv, int cus, DecodePlan* plan);
int64_t attn_decode_max_segments(int64_t max_req, int n_kv, int cus);
int64_t attn_decode_max_pieces(int64_t max_req, int64_t max_pages, int n_kv, int cus);
int attn_decode_record_floats();
void launch_attn_decode(int n_req, int n_pieces, const int32_t* work, const int32_t* cu_segs, int n_lanes,
                        const int32_t* lanes, const void* q, int64_t ldq, void* out, int64_t ldo,
                        const int32_t* req_slot, const int32_t* req_start, const int32_t* page_table, int max_pages,
                        const void* kpool, const void* vpool, int n_q, int n_kv, float* part,
                        const void* gate, hipStream_t st);

// Attention of each token's queries over its slot's cached keys 0..pos.
void launch_attn_paged(int act_fmt, int ntok, const void* q, int64_t ldq, void* out,
                       int64_t ldo, const int32_t* tok_slot, const int32_t* tok_pos,
                       const int32_t* page_table, int max_pages, const void* kpool,
                       const void* vpool, int n_q, int n_kv, int hd, const void* gate,
                       hipStream_t st);

// Prefill pooling: pool_sum[slot] = sum of the request's h rows; pooled[i] =
// [sum / n ; h[last]] (fp32; with pooled_bf16 != null also a bf16 hi/lo
// split: hi in rows [0, n), lo in rows [n, 2n)).
// cu_tiles[n_req + 1]: prefix sum of ceil(n_i / 32); part: [n_tiles, d] scratch.
void launch_pool_prefill(int n_req, int n_tiles, int d, int h_fmt, const void* h, int64_t ldh,
                         const int32_t* req_off, const int32_t* req_slot, const int32_t* cu_tiles,
                         float* part, float* pool_sum, float* pooled, uint16_t* pooled_bf16,
                         hipStream_t st);
// The final RMSNorm (x -> y2 fp32 and, if y is set, y in act format) fused
// with launch_pool_prefill on the normalised rows.  Rows are stored only
// when full_rows; otherwise only each request's last row of y2 is (all the
// pooling needs).  Returns false, launching nothing, for shapes the fused
// kernel does not take (d not 1024, 2048, 4096 or 8192, or misaligned).
bool launch_norm_pool_prefill(int act_fmt, int gamma_fmt, int n_req, int n_tiles, int d, const float* x,
                              int64_t ldx, const void* gamma, float eps, void* y, int64_t ldy, float* y2,
                              int64_t ldy2, bool full_rows, const int32_t* req_off, const int32_t* req_slot,
                              const int32_t* cu_tiles, float* part, float* pool_sum, float* pooled,
                              uint16_t* pooled_bf16, hipStream_t st);
// Decode step: final RMSNorm of x[i] (i = request) fused with its pooling;
// y (act) / y2 (f32) receive the normed rows when non-null.  Returns false,
// launching nothing, for shapes the fused kernel does not take (as
// launch_norm_pool_prefill).
// With rs (non-null; rowsum_supported(d)), row i is the RowSum's row i
// instead of x[i].
bool launch_norm_pool_step(int act_fmt, int gamma_fmt, int n_req, int d, const float* x, int64_t ldx,
                           const void* gamma, float eps, void* y, int64_t ldy, float* y2, int64_t ldy2,
                           const int32_t* req_slot, const int32_t* req_start, float* pool_sum, float* pooled,
                           uint16_t* pooled_bf16, hipStream_t st, const RowSum* rs = nullptr);
// Step pooling: pool_sum[slot] += h[i]; pooled[i] = [pool_sum / (start + 1) ; h[i]].
void launch_pool_step(int n_req, int d, int h_fmt, const void* h, int64_t ldh, const int32_t* req_slot,
                      const int32_t* req_start, float* pool_sum, float* pooled,
                      uint16_t* pooled_bf16, hipStream_t st);

// z[i] = w2 . relu(sum_s partial[s][i] + b1) + b2 (bf16 heads also add the
// lo-split rows partial[s][n + i])
void launch_head_finish(int w_fmt, int n_req, int h1, int splits, const float* partial,
                        const void* b1, const void* w2, const void* b2, float* z, hipStream_t st);

// Draft model head (Eq. 2): p[i] = softmax over v of logits row i (plus row
// n + i when two_rows: the hi/lo halves of a bf16-split input).
// stats: fp32 scratch of lm_softmax_stats_floats(n) floats (per-chunk max and sum).
int lm_softmax_stats_floats(int n);
void launch_lm_softmax(int n, int v, const float* logits, bool two_rows, float* stats, float* p, hipStream_t st);

void launch_copy_rows_act(int act_fmt, int rows, int d, const float* src, int64_t lds,
                          void* dst, int64_t ldd, hipStream_t st);

}  // namespace outlets
