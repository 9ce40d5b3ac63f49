// Row-wise kernels of the draft layer and the length head (HBM-bound):
// per-call token metadata, RMSNorm, rotary embedding + paged KV write,
// segmented mean/last pooling and the head's ReLU + final dot product.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace outlets {

namespace {

// The call's metadata block, written by the host into pinned host-coherent
// memory, copied into device memory together with the two things later
// kernels need from it first: the page-table updates (the (index, page)
// pairs after req_off | req_slot | req_start) and the per-token slot and
// position arrays.  One launch instead of a copy-engine transfer, whose
// completion the compute queue would wait on, and two kernels.  `host` is
// read with vector loads (it is not restrict-qualified), so nothing of it is
// kept in the scalar cache.
__global__ void __launch_bounds__(256)
meta_fetch_kernel(const int32_t* host, int count, int n_req, int n_pairs, int32_t* __restrict__ d_meta,
                  int32_t* __restrict__ page_table, int32_t* __restrict__ tok_slot, int32_t* __restrict__ tok_pos,
                  int32_t* __restrict__ last_idx) {
    const int tid = blockIdx.x * blockDim.x + threadIdx.x, nth = gridDim.x * blockDim.x;
    const int n4 = count / 4;
    const uint4* h4 = reinterpret_cast<const uint4*>(host);
    uint4* d4 = reinterpret_cast<uint4*>(d_meta);
    for (int i = tid; i < n4; i += nth) d4[i] = h4[i];
    for (int i = 4 * n4 + tid; i < count; i += nth) d_meta[i] = host[i];
    const int32_t* pairs = host + 3 * n_req + 1;
    for (int i = tid; i < n_pairs; i += nth) page_table[pairs[2 * i]] = pairs[2 * i + 1];
    for (int r = blockIdx.x; r < n_req; r += gridDim.x) {
        const int b = host[r], e = host[r + 1], slot = host[n_req + 1 + r], start = host[2 * n_req + 1 + r];
        for (int t = b + threadIdx.x; t < e; t += blockDim.x) {
            tok_slot[t] = slot;
            tok_pos[t] = start + (t - b);
        }
        if (threadIdx.x == 0) last_idx[r] = e - 1;
    }
}

// One 256-thread block per row.
template <typename TY, typename TG>
__global__ void __launch_bounds__(256)
rmsnorm_kernel(int d, const float* x, int64_t ldx, const TG* gamma, float eps, TY* y,
               int64_t ldy, float* y2, int64_t ldy2) {
    __shared__ float red[4];
    const int64_t row = blockIdx.x;
    const float* xr = x + row * ldx;
    float ss = 0.f;
    for (int c = threadIdx.x; c < d; c += 256) {
        float v = xr[c];
        ss = fmaf(v, v, ss);
    }
    ss = block_sum<256>(ss, red);
    const float inv = 1.0f / sqrtf(ss / d + eps);
    for (int c = threadIdx.x; c < d; c += 256) {
        float v = xr[c] * inv * load_act<TG>(gamma + c);
        if (y) store_act<TY>(y + row * ldy + c, v);
        if (y2) y2[row * ldy2 + c] = v;
    }
}

// Element group j4 (elements 4 j4 .. 4 j4 + 3) of a RowSum's row: the
// partials added in split order, then the residual added to that sum (the
// order of splitk_reduce), stored to rs.out when set.
__device__ __forceinline__ float4 rowsum_load(const RowSum& rs, int64_t row, int j4) {
    const float4* p = reinterpret_cast<const float4*>(rs.part + row * rs.ldp) + j4;
    const int64_t step = rs.plane / 4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int sp = 0; sp < rs.S; ++sp) {
        const float4 q = p[sp * step];
        v.x += q.x; v.y += q.y; v.z += q.z; v.w += q.w;
    }
    if (rs.resid) {
        const float4 r = reinterpret_cast<const float4*>(rs.resid + row * rs.ldr)[j4];
        v = make_float4(r.x + v.x, r.y + v.y, r.z + v.z, r.w + v.w);
    }
    if (rs.out) reinterpret_cast<float4*>(rs.out + row * rs.ldo)[j4] = v;
    return v;
}

// Vectorised form for d = 1024 V (V = 1..8 groups of 4 floats per thread):
// the row stays in registers between the sum of squares and the scaling,
// and every access is a 16-byte (x, y2) or 8-byte (bf16 y, gamma) access
// with consecutive threads on consecutive addresses.
// With SUM the row is a RowSum's (a split-K GEMM finished here) instead of x.
template <typename TY, typename TG, int V, bool SUM = false>
__global__ void __launch_bounds__(256)
rmsnorm_vec_kernel(int d, const float* x, int64_t ldx, const TG* gamma, float eps, TY* y,
                   int64_t ldy, float* y2, int64_t ldy2, RowSum rs = RowSum{}) {
    __shared__ float red[4];
    const int64_t row = blockIdx.x;
    const int t = threadIdx.x;
    const float4* xr = reinterpret_cast<const float4*>(x + row * ldx);
    float4 v[V];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < V; ++j) {
        v[j] = SUM ? rowsum_load(rs, row, j * 256 + t) : xr[j * 256 + t];
        ss = fmaf(v[j].x, v[j].x, fmaf(v[j].y, v[j].y, fmaf(v[j].z, v[j].z, fmaf(v[j].w, v[j].w, ss))));
    }
    ss = block_sum<256>(ss, red);
    const float inv = 1.0f / sqrtf(ss / d + eps);
#pragma unroll
    for (int j = 0; j < V; ++j) {
        const int c = (j * 256 + t) * 4;
        float g[4];
        if constexpr (sizeof(TG) == 4) {
            const float4 gv = *reinterpret_cast<const float4*>(gamma + c);
            g[0] = gv.x; g[1] = gv.y; g[2] = gv.z; g[3] = gv.w;
        } else {
            const uint2 gv = *reinterpret_cast<const uint2*>(gamma + c);
            g[0] = __uint_as_float(gv.x << 16); g[1] = __uint_as_float(gv.x & 0xffff0000u);
            g[2] = __uint_as_float(gv.y << 16); g[3] = __uint_as_float(gv.y & 0xffff0000u);
        }
        const float o0 = v[j].x * inv * g[0], o1 = v[j].y * inv * g[1];
        const float o2 = v[j].z * inv * g[2], o3 = v[j].w * inv * g[3];
        if (y) {
            if constexpr (sizeof(TY) == 4) {
                *reinterpret_cast<float4*>(y + row * ldy + c) = make_float4(o0, o1, o2, o3);
            } else {
                uint2 pk;
                pk.x = f32_to_bf16(o0) | (uint32_t(f32_to_bf16(o1)) << 16);
                pk.y = f32_to_bf16(o2) | (uint32_t(f32_to_bf16(o3)) << 16);
                *reinterpret_cast<uint2*>(y + row * ldy + c) = pk;
            }
        }
        if (y2) *reinterpret_cast<float4*>(y2 + row * ldy2 + c) = make_float4(o0, o1, o2, o3);
    }
}

// EAGLE-3 input embeddings: y[r] = RMSNorm(embed[tok[r]]) * gamma, one
// 256-thread block per row.  An id outside [0, vocab) reads nothing and
// gives a zero row.  V > 0: bf16 rows with d = 1024 V, four elements per
// thread and step (8-byte loads and stores); V = 0: any d and format.
template <typename TE, typename TG, int V>
__global__ void __launch_bounds__(256)
embed_norm_kernel(int d, int vocab, const int32_t* tok, const TE* embed, const TG* gamma, float eps,
                  TE* y, int64_t ldy) {
    __shared__ float red[4];
    const int64_t row = blockIdx.x;
    const int t = threadIdx.x;
    const int id = tok[row];
    const bool ok = id >= 0 && id < vocab;
    const TE* er = embed + (int64_t)(ok ? id : 0) * d;
    TE* yr = y + row * ldy;
    if constexpr (V > 0) {
        float v[V][4];
        float ss = 0.f;
#pragma unroll
        for (int j = 0; j < V; ++j) {
            const uint2 u = ok ? reinterpret_cast<const uint2*>(er)[j * 256 + t] : make_uint2(0u, 0u);
            v[j][0] = __uint_as_float(u.x << 16); v[j][1] = __uint_as_float(u.x & 0xffff0000u);
            v[j][2] = __uint_as_float(u.y << 16); v[j][3] = __uint_as_float(u.y & 0xffff0000u);
#pragma unroll
            for (int e = 0; e < 4; ++e) ss = fmaf(v[j][e], v[j][e], ss);
        }
        ss = block_sum<256>(ss, red);
        const float inv = ok ? 1.0f / sqrtf(ss / d + eps) : 0.f;
#pragma unroll
        for (int j = 0; j < V; ++j) {
            const int c = (j * 256 + t) * 4;
            float g[4];
            if constexpr (sizeof(TG) == 4) {
                const float4 gv = *reinterpret_cast<const float4*>(gamma + c);
                g[0] = gv.x; g[1] = gv.y; g[2] = gv.z; g[3] = gv.w;
            } else {
                const uint2 gv = *reinterpret_cast<const uint2*>(gamma + c);
                g[0] = __uint_as_float(gv.x << 16); g[1] = __uint_as_float(gv.x & 0xffff0000u);
                g[2] = __uint_as_float(gv.y << 16); g[3] = __uint_as_float(gv.y & 0xffff0000u);
            }
            uint2 pk;
            pk.x = f32_to_bf16(v[j][0] * inv * g[0]) | (uint32_t(f32_to_bf16(v[j][1] * inv * g[1])) << 16);
            pk.y = f32_to_bf16(v[j][2] * inv * g[2]) | (uint32_t(f32_to_bf16(v[j][3] * inv * g[3])) << 16);
            *reinterpret_cast<uint2*>(yr + c) = pk;
        }
    } else {
        float ss = 0.f;
        if (ok)
            for (int c = t; c < d; c += 256) {
                const float x = load_act<TE>(er + c);
                ss = fmaf(x, x, ss);
            }
        ss = block_sum<256>(ss, red);
        const float inv = ok ? 1.0f / sqrtf(ss / d + eps) : 0.f;
        for (int c = t; c < d; c += 256) {
            const float x = ok ? load_act<TE>(er + c) : 0.f;
            store_act<TE>(yr + c, x * inv * load_act<TG>(gamma + c));
        }
    }
}

// One block per token; thread work items are rotation pairs of the q and k
// heads and value elements.
template <typename T>
__global__ void __launch_bounds__(256)
rope_kv_kernel(T* qkv, int64_t ld, const int32_t* tok_slot, const int32_t* tok_pos,
               const int32_t* page_table, int max_pages, T* kpool, T* vpool,
               const float* cos_t, const float* sin_t, int n_q, int n_kv, int hd) {
    const int64_t t = blockIdx.x;
    const int pos = tok_pos[t], slot = tok_slot[t];
    const int half = hd / 2;
    const int page = page_table[(int64_t)slot * max_pages + pos / 16];
    const int off = pos % 16;
    T* row = qkv + t * ld;
    const float* cr = cos_t + (int64_t)pos * half;
    const float* sr = sin_t + (int64_t)pos * half;
    const int n_rot = (n_q + n_kv) * half;
    for (int w = threadIdx.x; w < n_rot; w += 256) {
        const int h = w / half, c = w % half;
        T* base = row + h * hd;
        const float x1 = load_act<T>(base + c), x2 = load_act<T>(base + c + half);
        const float cs = cr[c], sn = sr[c];
        const float y1 = x1 * cs - x2 * sn, y2 = x2 * cs + x1 * sn;
        if (h < n_q) {
            store_act<T>(base + c, y1);
            store_act<T>(base + c + half, y2);
        } else {
            const int g = h - n_q;
            T* dst = kpool + (((int64_t)page * n_kv + g) * 16 + off) * hd;
            store_act<T>(dst + c, y1);
            store_act<T>(dst + c + half, y2);
        }
    }
    // value pages are stored transposed, [n_kv][hd][16 tokens], so that a
    // channel's 16 values of a page are contiguous
    const T* vrow = row + (n_q + n_kv) * hd;
    for (int w = threadIdx.x; w < n_kv * hd; w += 256) {
        const int g = w / hd, c = w % hd;
        vpool[(((int64_t)page * n_kv + g) * hd + c) * 16 + off] = vrow[w];
    }
}

// bf16 form: one wave per token, four rotation pairs per lane and step
// (8-byte loads and stores of the two halves, 16-byte cos/sin loads).
__global__ void __launch_bounds__(256)
rope_kv_bf16_kernel(int ntok, bf16_t* qkv, int64_t ld, const int32_t* tok_slot, const int32_t* tok_pos,
                    const int32_t* page_table, int max_pages, bf16_t* kpool, bf16_t* vpool,
                    const float* cos_t, const float* sin_t, int n_q, int n_kv, int hd) {
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= ntok) return;
    const int lane = threadIdx.x & 63;
    const int pos = tok_pos[t], slot = tok_slot[t];
    const int half = hd / 2, quads = half / 4;
    const int page = page_table[(int64_t)slot * max_pages + pos / 16];
    const int off = pos % 16;
    bf16_t* row = qkv + t * ld;
    const float* cr = cos_t + (int64_t)pos * half;
    const float* sr = sin_t + (int64_t)pos * half;
    const int n_items = (n_q + n_kv) * quads;
    for (int w = lane; w < n_items; w += 64) {
        const int h = w / quads, c = (w % quads) * 4;
        bf16_t* base = row + h * hd;
        const uint2 a1 = *reinterpret_cast<const uint2*>(base + c);
        const uint2 a2 = *reinterpret_cast<const uint2*>(base + c + half);
        const float4 cs = *reinterpret_cast<const float4*>(cr + c);
        const float4 sn = *reinterpret_cast<const float4*>(sr + c);
        const float x1[4] = {__uint_as_float(a1.x << 16), __uint_as_float(a1.x & 0xffff0000u),
                             __uint_as_float(a1.y << 16), __uint_as_float(a1.y & 0xffff0000u)};
        const float x2[4] = {__uint_as_float(a2.x << 16), __uint_as_float(a2.x & 0xffff0000u),
                             __uint_as_float(a2.y << 16), __uint_as_float(a2.y & 0xffff0000u)};
        const float cv[4] = {cs.x, cs.y, cs.z, cs.w}, sv[4] = {sn.x, sn.y, sn.z, sn.w};
        uint16_t y1[4], y2[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            y1[e] = f32_to_bf16(x1[e] * cv[e] - x2[e] * sv[e]);
            y2[e] = f32_to_bf16(x2[e] * cv[e] + x1[e] * sv[e]);
        }
        const uint2 o1 = make_uint2(y1[0] | (uint32_t(y1[1]) << 16), y1[2] | (uint32_t(y1[3]) << 16));
        const uint2 o2 = make_uint2(y2[0] | (uint32_t(y2[1]) << 16), y2[2] | (uint32_t(y2[3]) << 16));
        bf16_t* dst = h < n_q ? base : kpool + (((int64_t)page * n_kv + (h - n_q)) * 16 + off) * hd;
        *reinterpret_cast<uint2*>(dst + c) = o1;
        *reinterpret_cast<uint2*>(dst + c + half) = o2;
    }
    const bf16_t* vrow = row + (n_q + n_kv) * hd;
    for (int w = lane; w < n_kv * hd; w += 64) {
        const int g = w / hd, c = w % hd;
        vpool[(((int64_t)page * n_kv + g) * hd + c) * 16 + off] = vrow[w];
    }
}

// The head's MFMA GEMM reads bf16: an fp32 value v is passed as two rows,
// hi = bf16(v) in row i and lo = bf16(v - hi) in row n + i (n = requests),
// whose products the head sums, so the head input keeps ~16 mantissa bits.
__device__ __forceinline__ void split_bf16(float v, uint16_t* hi_row, int64_t lo_offset) {
    const bf16_t hi = f32_to_bf16(v);
    hi_row[0] = hi;
    hi_row[lo_offset] = f32_to_bf16(v - bf16_to_f32(hi));
}

// Prefill pooling in two deterministic stages.  Stage 1, grid (tiles,
// ceil(d / 256)): tile t (request r's rows [32 k, 32 k + 32), t = cu_tiles[r]
// + k) sums its rows in order.  Stage 2, grid (n_req, ceil(d / 256)): each
// request sums its tiles in order.  Tiles are relative to the request start,
// so the result does not depend on the rest of the batch.
template <typename TH>
__global__ void __launch_bounds__(256)
pool_tiles_kernel(int d, int n_req, const TH* h, int64_t ldh, const int32_t* req_off,
                  const int32_t* cu_tiles, float* part) {
    const int t = blockIdx.x;
    const int c = blockIdx.y * 256 + threadIdx.x;
    if (c >= d) return;
    int lo = 0, hi = n_req - 1;        // request r with cu_tiles[r] <= t < cu_tiles[r + 1]
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (cu_tiles[mid] <= t) lo = mid; else hi = mid - 1;
    }
    const int b = req_off[lo] + (t - cu_tiles[lo]) * 32;
    const int e = min(b + 32, req_off[lo + 1]);
    // rows summed in order; their loads are issued eight at a time (one
    // dependent load per row measured 2.3 TB/s on a 237 MB bf16 state)
    float s = 0.f;
    int r = b;
    for (; r + 8 <= e; r += 8) {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = load_act<TH>(h + (int64_t)(r + j) * ldh + c);
#pragma unroll
        for (int j = 0; j < 8; ++j) s += v[j];
    }
    for (; r < e; ++r) s += load_act<TH>(h + (int64_t)r * ldh + c);
    part[(int64_t)t * d + c] = s;
}

// The final RMSNorm fused with stage 1 of the prefill pooling (d = 1024 V):
// tile t (as in pool_tiles_kernel) normalises its rows in order with the
// arithmetic of rmsnorm_vec_kernel and sums them in row order into part[t],
// so the sums are those of the unfused pair, bit for bit.  Normalised rows
// are stored (y2 fp32, y in the act format) only when full_rows; otherwise
// only each request's last row, which the head input also needs.  The next
// row's loads are issued before the current row's reduction.
template <typename TY, typename TG, int V>
__global__ void __launch_bounds__(256)
norm_pool_tiles_kernel(int d, int n_req, const float* x, int64_t ldx, const TG* gamma, float eps, TY* y,
                       int64_t ldy, float* y2, int64_t ldy2, int full_rows, const int32_t* req_off,
                       const int32_t* cu_tiles, float* part) {
    __shared__ float red[4];
    const int t = blockIdx.x, th = threadIdx.x;
    int lo = 0, hi = n_req - 1;        // request lo with cu_tiles[lo] <= t < cu_tiles[lo + 1]
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (cu_tiles[mid] <= t) lo = mid; else hi = mid - 1;
    }
    const int b = req_off[lo] + (t - cu_tiles[lo]) * 32;
    const int e = min(b + 32, req_off[lo + 1]);
    const int last = req_off[lo + 1] - 1;
    float g[V][4];
#pragma unroll
    for (int j = 0; j < V; ++j) {
        const int c = (j * 256 + th) * 4;
        if constexpr (sizeof(TG) == 4) {
            const float4 gv = *reinterpret_cast<const float4*>(gamma + c);
            g[j][0] = gv.x; g[j][1] = gv.y; g[j][2] = gv.z; g[j][3] = gv.w;
        } else {
            const uint2 gv = *reinterpret_cast<const uint2*>(gamma + c);
            g[j][0] = __uint_as_float(gv.x << 16); g[j][1] = __uint_as_float(gv.x & 0xffff0000u);
            g[j][2] = __uint_as_float(gv.y << 16); g[j][3] = __uint_as_float(gv.y & 0xffff0000u);
        }
    }
    float4 acc[V], vn[V];
#pragma unroll
    for (int j = 0; j < V; ++j) {
        acc[j] = make_float4(0.f, 0.f, 0.f, 0.f);
        vn[j] = reinterpret_cast<const float4*>(x + (int64_t)b * ldx)[j * 256 + th];
    }
    for (int r = b; r < e; ++r) {
        float4 v[V];
        float ss = 0.f;
#pragma unroll
        for (int j = 0; j < V; ++j) {
            v[j] = vn[j];
            ss = fmaf(v[j].x, v[j].x, fmaf(v[j].y, v[j].y, fmaf(v[j].z, v[j].z, fmaf(v[j].w, v[j].w, ss))));
        }
        if (r + 1 < e) {
#pragma unroll
            for (int j = 0; j < V; ++j) vn[j] = reinterpret_cast<const float4*>(x + (int64_t)(r + 1) * ldx)[j * 256 + th];
        }
        ss = block_sum<256>(ss, red);
        const float inv = 1.0f / sqrtf(ss / d + eps);
        const bool store = full_rows || r == last;
#pragma unroll
        for (int j = 0; j < V; ++j) {
            const int c = (j * 256 + th) * 4;
            const float o0 = v[j].x * inv * g[j][0], o1 = v[j].y * inv * g[j][1];
            const float o2 = v[j].z * inv * g[j][2], o3 = v[j].w * inv * g[j][3];
            acc[j].x += o0; acc[j].y += o1; acc[j].z += o2; acc[j].w += o3;
            if (store) {
                if (y) {
                    if constexpr (sizeof(TY) == 4) {
                        *reinterpret_cast<float4*>(y + (int64_t)r * ldy + c) = make_float4(o0, o1, o2, o3);
                    } else {
                        uint2 pk;
                        pk.x = f32_to_bf16(o0) | (uint32_t(f32_to_bf16(o1)) << 16);
                        pk.y = f32_to_bf16(o2) | (uint32_t(f32_to_bf16(o3)) << 16);
                        *reinterpret_cast<uint2*>(y + (int64_t)r * ldy + c) = pk;
                    }
                }
                *reinterpret_cast<float4*>(y2 + (int64_t)r * ldy2 + c) = make_float4(o0, o1, o2, o3);
            }
        }
    }
#pragma unroll
    for (int j = 0; j < V; ++j) reinterpret_cast<float4*>(part + (int64_t)t * d)[j * 256 + th] = acc[j];
}

template <typename TH>
__global__ void __launch_bounds__(256)
pool_prefill_kernel(int d, const TH* h, int64_t ldh, const int32_t* req_off,
                    const int32_t* req_slot, const int32_t* cu_tiles, const float* part,
                    float* pool_sum, float* pooled, uint16_t* pooled_bf16) {
    const int i = blockIdx.x;
    const int c = blockIdx.y * 256 + threadIdx.x;
    if (c >= d) return;
    const int b = req_off[i], e = req_off[i + 1];
    // tile sums added in tile order; their loads are issued eight at a time
    // (one dependent load per tile took 39 us for a 32-request, 28,944-token
    // batch whose longest prompt has 128 tiles)
    float s = 0.f;
    int t = cu_tiles[i];
    const int t1 = cu_tiles[i + 1];
    for (; t + 8 <= t1; t += 8) {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = part[(int64_t)(t + j) * d + c];
#pragma unroll
        for (int j = 0; j < 8; ++j) s += v[j];
    }
    for (; t < t1; ++t) s += part[(int64_t)t * d + c];
    pool_sum[(int64_t)req_slot[i] * d + c] = s;
    const float mean = s / static_cast<float>(e - b);
    const float last = load_act<TH>(h + (int64_t)(e - 1) * ldh + c);
    pooled[(int64_t)i * 2 * d + c] = mean;
    pooled[(int64_t)i * 2 * d + d + c] = last;
    if (pooled_bf16) {
        split_bf16(mean, pooled_bf16 + (int64_t)i * 2 * d + c, (int64_t)gridDim.x * 2 * d);
        split_bf16(last, pooled_bf16 + (int64_t)i * 2 * d + d + c, (int64_t)gridDim.x * 2 * d);
    }
}

template <typename TH>
__global__ void __launch_bounds__(256)
pool_step_kernel(int d, const TH* h, int64_t ldh, const int32_t* req_slot,
                 const int32_t* req_start, float* pool_sum, float* pooled, uint16_t* pooled_bf16) {
    const int i = blockIdx.x;
    const int c = blockIdx.y * 256 + threadIdx.x;
    if (c >= d) return;
    const float x = load_act<TH>(h + (int64_t)i * ldh + c);
    float* ps = pool_sum + (int64_t)req_slot[i] * d + c;
    const float s = *ps + x;
    *ps = s;
    const float mean = s / static_cast<float>(req_start[i] + 1);
    pooled[(int64_t)i * 2 * d + c] = mean;
    pooled[(int64_t)i * 2 * d + d + c] = x;
    if (pooled_bf16) {
        split_bf16(mean, pooled_bf16 + (int64_t)i * 2 * d + c, (int64_t)gridDim.x * 2 * d);
        split_bf16(x, pooled_bf16 + (int64_t)i * 2 * d + d + c, (int64_t)gridDim.x * 2 * d);
    }
}

// Decode step: final RMSNorm of request i's new row x[i] and its pooling in
// one pass: one block of NT threads per request, V float4 per thread (NT V =
// d / 4; the few rows of a step need wide blocks to keep the CUs busy).  The
// scaling and the pooling arithmetic are rmsnorm_vec_kernel's and
// pool_step_kernel's; the sum of squares is taken over NT partial sums.
// y / y2 (the h_draft row) are stored only when non-null.
template <typename TY, typename TG, int NT, int V, bool SUM = false>
__global__ void __launch_bounds__(NT)
norm_pool_step_kernel(int d, int n_req, const float* x, int64_t ldx, const TG* gamma, float eps, TY* y,
                      int64_t ldy, float* y2, int64_t ldy2, const int32_t* req_slot, const int32_t* req_start,
                      float* pool_sum, float* pooled, uint16_t* pooled_bf16, RowSum rs = RowSum{}) {
    __shared__ float red[NT / 64];
    const int64_t row = blockIdx.x;
    const int t = threadIdx.x;
    const float4* xr = reinterpret_cast<const float4*>(x + row * ldx);
    float4 v[V];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < V; ++j) {
        v[j] = SUM ? rowsum_load(rs, row, j * NT + t) : xr[j * NT + t];
        ss = fmaf(v[j].x, v[j].x, fmaf(v[j].y, v[j].y, fmaf(v[j].z, v[j].z, fmaf(v[j].w, v[j].w, ss))));
    }
    ss = block_sum<NT>(ss, red);
    const float inv = 1.0f / sqrtf(ss / d + eps);
    float* ps = pool_sum + (int64_t)req_slot[row] * d;
    const float cnt = static_cast<float>(req_start[row] + 1);
    float* prow = pooled + row * 2 * d;
    const int64_t lo = (int64_t)n_req * 2 * d;
#pragma unroll
    for (int j = 0; j < V; ++j) {
        const int c = (j * NT + t) * 4;
        float g[4];
        if constexpr (sizeof(TG) == 4) {
            const float4 gv = *reinterpret_cast<const float4*>(gamma + c);
            g[0] = gv.x; g[1] = gv.y; g[2] = gv.z; g[3] = gv.w;
        } else {
            const uint2 gv = *reinterpret_cast<const uint2*>(gamma + c);
            g[0] = __uint_as_float(gv.x << 16); g[1] = __uint_as_float(gv.x & 0xffff0000u);
            g[2] = __uint_as_float(gv.y << 16); g[3] = __uint_as_float(gv.y & 0xffff0000u);
        }
        const float o[4] = {v[j].x * inv * g[0], v[j].y * inv * g[1], v[j].z * inv * g[2], v[j].w * inv * g[3]};
        if (y) {
            if constexpr (sizeof(TY) == 4) {
                *reinterpret_cast<float4*>(y + row * ldy + c) = make_float4(o[0], o[1], o[2], o[3]);
            } else {
                uint2 pk;
                pk.x = f32_to_bf16(o[0]) | (uint32_t(f32_to_bf16(o[1])) << 16);
                pk.y = f32_to_bf16(o[2]) | (uint32_t(f32_to_bf16(o[3])) << 16);
                *reinterpret_cast<uint2*>(y + row * ldy + c) = pk;
            }
        }
        if (y2) *reinterpret_cast<float4*>(y2 + row * ldy2 + c) = make_float4(o[0], o[1], o[2], o[3]);
        const float4 s0 = *reinterpret_cast<const float4*>(ps + c);
        const float s[4] = {s0.x + o[0], s0.y + o[1], s0.z + o[2], s0.w + o[3]};
        *reinterpret_cast<float4*>(ps + c) = make_float4(s[0], s[1], s[2], s[3]);
        const float mean[4] = {s[0] / cnt, s[1] / cnt, s[2] / cnt, s[3] / cnt};
        *reinterpret_cast<float4*>(prow + c) = make_float4(mean[0], mean[1], mean[2], mean[3]);
        *reinterpret_cast<float4*>(prow + d + c) = make_float4(o[0], o[1], o[2], o[3]);
        if (pooled_bf16) {
            uint16_t hm[4], lm[4], hx[4], lx[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                hm[e] = f32_to_bf16(mean[e]);
                lm[e] = f32_to_bf16(mean[e] - bf16_to_f32(hm[e]));
                hx[e] = f32_to_bf16(o[e]);
                lx[e] = f32_to_bf16(o[e] - bf16_to_f32(hx[e]));
            }
            uint16_t* pb = pooled_bf16 + row * 2 * d + c;
            auto pack = [](const uint16_t* h) {
                return make_uint2(h[0] | (uint32_t(h[1]) << 16), h[2] | (uint32_t(h[3]) << 16));
            };
            *reinterpret_cast<uint2*>(pb) = pack(hm);
            *reinterpret_cast<uint2*>(pb + lo) = pack(lm);
            *reinterpret_cast<uint2*>(pb + d) = pack(hx);
            *reinterpret_cast<uint2*>(pb + d + lo) = pack(lx);
        }
    }
}

template <typename TW>
__global__ void __launch_bounds__(256)
head_finish_kernel(int h1, int splits, int n_req, int rows, const float* partial, const TW* b1,
                   const TW* w2, const TW* b2, float* z) {
    __shared__ float red[4];
    const int i = blockIdx.x;
    float acc = 0.f;
    for (int j = threadIdx.x; j < h1; j += 256) {
        float v = load_act<TW>(b1 + j);
        for (int s = 0; s < splits; ++s) {
            v += partial[((int64_t)s * rows + i) * h1 + j];
            if (rows > n_req) v += partial[((int64_t)s * rows + n_req + i) * h1 + j];
        }
        acc = fmaf(fmaxf(v, 0.f), load_act<TW>(w2 + j), acc);
    }
    acc = block_sum<256>(acc, red);
    if (threadIdx.x == 0) z[i] = acc + load_act<TW>(b2);
}

// Same result for a split count that is a multiple of S and h1 a multiple of
// 4: each thread takes four consecutive hidden units and, per group of S
// splits, issues all 2 S of its partial loads (16-byte) before summing them
// in split order, so the block waits out one memory latency per group
// instead of one per split.
template <typename TW, int S>
__global__ void __launch_bounds__(256)
head_finish_vec_kernel(int h1, int n_req, int rows, int splits, const float* partial, const TW* b1,
                       const TW* w2, const TW* b2, float* z) {
    __shared__ float red[4];
    const int i = blockIdx.x;
    const bool lo = rows > n_req;
    float acc = 0.f;
    for (int j = threadIdx.x * 4; j < h1; j += 1024) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = load_act<TW>(b1 + j + e);
        // splits in groups of S (loads of a group issued together), summed in order
        for (int s0 = 0; s0 < splits; s0 += S) {
            float4 ph[S], pl[S];
#pragma unroll
            for (int q = 0; q < S; ++q) {
                const int64_t sp = s0 + q;
                ph[q] = *reinterpret_cast<const float4*>(partial + (sp * rows + i) * h1 + j);
                pl[q] = lo ? *reinterpret_cast<const float4*>(partial + (sp * rows + n_req + i) * h1 + j)
                           : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
            for (int q = 0; q < S; ++q) {
                v[0] += ph[q].x; v[1] += ph[q].y; v[2] += ph[q].z; v[3] += ph[q].w;
                if (lo) { v[0] += pl[q].x; v[1] += pl[q].y; v[2] += pl[q].z; v[3] += pl[q].w; }
            }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) acc = fmaf(fmaxf(v[e], 0.f), load_act<TW>(w2 + j + e), acc);
    }
    acc = block_sum<256>(acc, red);
    if (threadIdx.x == 0) z[i] = acc + load_act<TW>(b2);
}

template <typename T>
__global__ void copy_rows_kernel(int d, const float* src, int64_t lds, T* dst, int64_t ldd) {
    const int64_t r = blockIdx.x;
    for (int c = threadIdx.x; c < d; c += blockDim.x) store_act<T>(dst + r * ldd + c, src[r * lds + c]);
}

}  // namespace

void launch_meta_fetch(const int32_t* host_meta, int count, int n_req, int n_pairs, int32_t* d_meta,
                       int32_t* page_table, int32_t* tok_slot, int32_t* tok_pos, int32_t* last_idx, hipStream_t st) {
    if (count <= 0) return;
    const int blocks = std::max(1, std::max(n_req, (count / 4 + 255) / 256));
    hipLaunchKernelGGL(meta_fetch_kernel, dim3(blocks), dim3(256), 0, st, host_meta, count, n_req, n_pairs, d_meta,
                       page_table, tok_slot, tok_pos, last_idx);
}

bool rowsum_supported(int d) { return d == 1024 || d == 2048 || d == 4096 || d == 8192; }

void launch_rmsnorm_sum(int act_fmt, int gamma_fmt, int rows, int d, const RowSum& rs, const void* gamma,
                        float eps, void* y, int64_t ldy, hipStream_t st) {
    if (rows <= 0) return;
    const int V = d / 1024;
#define OUTLETS_NORMS_V(TY, TG)                                                                            \
    switch (V) {                                                                                           \
        case 1: hipLaunchKernelGGL((rmsnorm_vec_kernel<TY, TG, 1, true>), dim3(rows), dim3(256), 0, st, d, nullptr, 0, \
                                   static_cast<const TG*>(gamma), eps, static_cast<TY*>(y), ldy, nullptr, 0, rs); break; \
        case 2: hipLaunchKernelGGL((rmsnorm_vec_kernel<TY, TG, 2, true>), dim3(rows), dim3(256), 0, st, d, nullptr, 0, \
                                   static_cast<const TG*>(gamma), eps, static_cast<TY*>(y), ldy, nullptr, 0, rs); break; \
        case 4: hipLaunchKernelGGL((rmsnorm_vec_kernel<TY, TG, 4, true>), dim3(rows), dim3(256), 0, st, d, nullptr, 0, \
                                   static_cast<const TG*>(gamma), eps, static_cast<TY*>(y), ldy, nullptr, 0, rs); break; \
        case 8: hipLaunchKernelGGL((rmsnorm_vec_kernel<TY, TG, 8, true>), dim3(rows), dim3(256), 0, st, d, nullptr, 0, \
                                   static_cast<const TG*>(gamma), eps, static_cast<TY*>(y), ldy, nullptr, 0, rs); break; \
    }
    if (act_fmt == FMT_F32) { OUTLETS_NORMS_V(float, float) }
    else if (gamma_fmt == FMT_F32) { OUTLETS_NORMS_V(bf16_t, float) }
    else { OUTLETS_NORMS_V(bf16_t, bf16_t) }
#undef OUTLETS_NORMS_V
}

void launch_rmsnorm(int act_fmt, int gamma_fmt, int rows, int d, const float* x, int64_t ldx,
                    const void* gamma, float eps, void* y, int64_t ldy, float* y2,
                    int64_t ldy2, hipStream_t st) {
    if (rows <= 0) return;
    // vectorised path: d a multiple of 1024 up to 8192, 16-byte aligned rows
    const bool vec = d % 1024 == 0 && d <= 8192 && ldx % 4 == 0 && (!y || ldy % 4 == 0) &&
                     (!y2 || ldy2 % 4 == 0) && reinterpret_cast<uintptr_t>(x) % 16 == 0 &&
                     (!y || reinterpret_cast<uintptr_t>(y) % 16 == 0) &&
                     (!y2 || reinterpret_cast<uintptr_t>(y2) % 16 == 0) &&
                     reinterpret_cast<uintptr_t>(gamma) % 16 == 0;
    if (vec) {
        const int V = d / 1024;
#define OUTLETS_NORM_V(TY, TG)                                                                  \
    switch (V) {                                                                                \
        case 1: hipLaunchKernelGGL((rmsnorm_vec_kernel<TY, TG, 1>), dim3(rows), dim3(256), 0, st, d, x, ldx, \
                                   static_cast<const TG*>(gamma), eps, static_cast<TY*>(y), ldy, y2, ldy2); break; \
        case 2: hipLaunchKernelGGL((rmsnorm_vec_kernel<TY, TG, 2>), dim3(rows), dim3(256), 0, st, d, x, ldx, \
                                   static_cast<const TG*>(gamma), eps, static_cast<TY*>(y), ldy, y2, ldy2); break; \
        case 4: hipLaunchKernelGGL((rmsnorm_vec_kernel<TY, TG, 4>), dim3(rows), dim3(256), 0, st, d, x, ldx, \
                                   static_cast<const TG*>(gamma), eps, static_cast<TY*>(y), ldy, y2, ldy2); break; \
        case 8: hipLaunchKernelGGL((rmsnorm_vec_kernel<TY, TG, 8>), dim3(rows), dim3(256), 0, st, d, x, ldx, \
                                   static_cast<const TG*>(gamma), eps, static_cast<TY*>(y), ldy, y2, ldy2); break; \
        default: goto scalar;                                                                   \
    }
        if (act_fmt == FMT_F32) { OUTLETS_NORM_V(float, float) }
        else if (gamma_fmt == FMT_F32) { OUTLETS_NORM_V(bf16_t, float) }
        else { OUTLETS_NORM_V(bf16_t, bf16_t) }
#undef OUTLETS_NORM_V
        return;
    }
scalar:
    if (act_fmt == FMT_F32) {
        hipLaunchKernelGGL((rmsnorm_kernel<float, float>), dim3(rows), dim3(256), 0, st, d, x, ldx,
                           static_cast<const float*>(gamma), eps, static_cast<float*>(y), ldy, y2, ldy2);
    } else if (gamma_fmt == FMT_F32) {
        hipLaunchKernelGGL((rmsnorm_kernel<bf16_t, float>), dim3(rows), dim3(256), 0, st, d, x, ldx,
                           static_cast<const float*>(gamma), eps, static_cast<bf16_t*>(y), ldy, y2, ldy2);
    } else {
        hipLaunchKernelGGL((rmsnorm_kernel<bf16_t, bf16_t>), dim3(rows), dim3(256), 0, st, d, x, ldx,
                           static_cast<const bf16_t*>(gamma), eps, static_cast<bf16_t*>(y), ldy, y2, ldy2);
    }
}

void launch_embed_norm(int act_fmt, int gamma_fmt, int rows, int d, int vocab, const int32_t* tok,
                       const void* embed, const void* gamma, float eps, void* y, int64_t ldy,
                       hipStream_t st) {
    if (rows <= 0) return;
    const dim3 grid(rows), blk(256);
    if (act_fmt == FMT_F32) {
        hipLaunchKernelGGL((embed_norm_kernel<float, float, 0>), grid, blk, 0, st, d, vocab, tok,
                           static_cast<const float*>(embed), static_cast<const float*>(gamma), eps,
                           static_cast<float*>(y), ldy);
        return;
    }
    const bool vec = d % 1024 == 0 && d <= 8192 && ldy % 4 == 0 &&
                     reinterpret_cast<uintptr_t>(embed) % 8 == 0 && reinterpret_cast<uintptr_t>(y) % 8 == 0 &&
                     reinterpret_cast<uintptr_t>(gamma) % 16 == 0;
    const int V = vec ? d / 1024 : 0;
#define OUTLETS_EMB(TG, VV)                                                                        \
    hipLaunchKernelGGL((embed_norm_kernel<bf16_t, TG, VV>), grid, blk, 0, st, d, vocab, tok,      \
                       static_cast<const bf16_t*>(embed), static_cast<const TG*>(gamma), eps,     \
                       static_cast<bf16_t*>(y), ldy)
#define OUTLETS_EMB_G(TG)                                       \
    switch (V) {                                                \
        case 1: OUTLETS_EMB(TG, 1); break;                      \
        case 2: OUTLETS_EMB(TG, 2); break;                      \
        case 4: OUTLETS_EMB(TG, 4); break;                      \
        case 8: OUTLETS_EMB(TG, 8); break;                      \
        default: OUTLETS_EMB(TG, 0); break;                     \
    }
    if (gamma_fmt == FMT_F32) { OUTLETS_EMB_G(float) }
    else { OUTLETS_EMB_G(bf16_t) }
#undef OUTLETS_EMB_G
#undef OUTLETS_EMB
}

void launch_rope_kv(int act_fmt, int ntok, void* qkv, int64_t ld, const int32_t* tok_slot,
                    const int32_t* tok_pos, const int32_t* page_table, int max_pages,
                    void* kpool, void* vpool, const float* cos_t, const float* sin_t,
                    int n_q, int n_kv, int hd, hipStream_t st) {
    if (ntok <= 0) return;
    if (act_fmt == FMT_F32)
        hipLaunchKernelGGL((rope_kv_kernel<float>), dim3(ntok), dim3(256), 0, st,
                           static_cast<float*>(qkv), ld, tok_slot, tok_pos, page_table, max_pages,
                           static_cast<float*>(kpool), static_cast<float*>(vpool), cos_t, sin_t,
                           n_q, n_kv, hd);
    else if (hd % 8 == 0 && ld % 4 == 0 && reinterpret_cast<uintptr_t>(qkv) % 8 == 0)
        hipLaunchKernelGGL(rope_kv_bf16_kernel, dim3((ntok + 3) / 4), dim3(256), 0, st, ntok,
                           static_cast<bf16_t*>(qkv), ld, tok_slot, tok_pos, page_table, max_pages,
                           static_cast<bf16_t*>(kpool), static_cast<bf16_t*>(vpool), cos_t, sin_t,
                           n_q, n_kv, hd);
    else
        hipLaunchKernelGGL((rope_kv_kernel<bf16_t>), dim3(ntok), dim3(256), 0, st,
                           static_cast<bf16_t*>(qkv), ld, tok_slot, tok_pos, page_table, max_pages,
                           static_cast<bf16_t*>(kpool), static_cast<bf16_t*>(vpool), cos_t, sin_t,
                           n_q, n_kv, hd);
}

void launch_pool_prefill(int n_req, int n_tiles, int d, int h_fmt, const void* h, int64_t ldh,
                         const int32_t* req_off, const int32_t* req_slot, const int32_t* cu_tiles,
                         float* part, float* pool_sum, float* pooled, uint16_t* pooled_bf16,
                         hipStream_t st) {
    if (n_req <= 0) return;
    const dim3 gt(n_tiles, (d + 255) / 256), gr(n_req, (d + 255) / 256);
    if (h_fmt == FMT_F32) {
        const float* hh = static_cast<const float*>(h);
        hipLaunchKernelGGL(pool_tiles_kernel<float>, gt, dim3(256), 0, st, d, n_req, hh, ldh, req_off, cu_tiles, part);
        hipLaunchKernelGGL(pool_prefill_kernel<float>, gr, dim3(256), 0, st, d, hh, ldh, req_off, req_slot,
                           cu_tiles, part, pool_sum, pooled, pooled_bf16);
    } else {
        const bf16_t* hh = static_cast<const bf16_t*>(h);
        hipLaunchKernelGGL(pool_tiles_kernel<bf16_t>, gt, dim3(256), 0, st, d, n_req, hh, ldh, req_off, cu_tiles, part);
        hipLaunchKernelGGL(pool_prefill_kernel<bf16_t>, gr, dim3(256), 0, st, d, hh, ldh, req_off, req_slot,
                           cu_tiles, part, pool_sum, pooled, pooled_bf16);
    }
}

bool launch_norm_pool_prefill(int act_fmt, int gamma_fmt, int n_req, int n_tiles, int d, const float* x,
                              int64_t ldx, const void* gamma, float eps, void* y, int64_t ldy, float* y2,
                              int64_t ldy2, bool full_rows, const int32_t* req_off, const int32_t* req_slot,
                              const int32_t* cu_tiles, float* part, float* pool_sum, float* pooled,
                              uint16_t* pooled_bf16, hipStream_t st) {
    const bool vec = d % 1024 == 0 && d <= 8192 && ldx % 4 == 0 && (!y || ldy % 4 == 0) && ldy2 % 4 == 0 &&
                     reinterpret_cast<uintptr_t>(x) % 16 == 0 && reinterpret_cast<uintptr_t>(y) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(y2) % 16 == 0 && reinterpret_cast<uintptr_t>(gamma) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(part) % 16 == 0 && (d / 1024 & (d / 1024 - 1)) == 0;
    if (!vec) return false;
    if (n_req <= 0) return true;
    const int V = d / 1024, fr = full_rows ? 1 : 0;
#define OUTLETS_NP_V(TY, TG, VV)                                                                        \
    case VV:                                                                                            \
        hipLaunchKernelGGL((norm_pool_tiles_kernel<TY, TG, VV>), dim3(n_tiles), dim3(256), 0, st, d, n_req, x, \
                           ldx, static_cast<const TG*>(gamma), eps, static_cast<TY*>(y), ldy, y2, ldy2, fr,  \
                           req_off, cu_tiles, part);                                                    \
        break;
#define OUTLETS_NP(TY, TG)                                                                              \
    switch (V) { OUTLETS_NP_V(TY, TG, 1) OUTLETS_NP_V(TY, TG, 2) OUTLETS_NP_V(TY, TG, 4) OUTLETS_NP_V(TY, TG, 8) }
    if (act_fmt == FMT_F32) { OUTLETS_NP(float, float) }
    else if (gamma_fmt == FMT_F32) { OUTLETS_NP(bf16_t, float) }
    else { OUTLETS_NP(bf16_t, bf16_t) }
#undef OUTLETS_NP
#undef OUTLETS_NP_V
    const dim3 gr(n_req, (d + 255) / 256);
    hipLaunchKernelGGL(pool_prefill_kernel<float>, gr, dim3(256), 0, st, d, static_cast<const float*>(y2), ldy2,
                       req_off, req_slot, cu_tiles, part, pool_sum, pooled, pooled_bf16);
    return true;
}

bool launch_norm_pool_step(int act_fmt, int gamma_fmt, int n_req, int d, const float* x, int64_t ldx,
                           const void* gamma, float eps, void* y, int64_t ldy, float* y2, int64_t ldy2,
                           const int32_t* req_slot, const int32_t* req_start, float* pool_sum, float* pooled,
                           uint16_t* pooled_bf16, hipStream_t st, const RowSum* rs) {
    const bool vec = d % 1024 == 0 && d <= 8192 && ldx % 4 == 0 && (!y || ldy % 4 == 0) && (!y2 || ldy2 % 4 == 0) &&
                     reinterpret_cast<uintptr_t>(x) % 16 == 0 && reinterpret_cast<uintptr_t>(y) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(y2) % 16 == 0 && reinterpret_cast<uintptr_t>(gamma) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(pool_sum) % 16 == 0 && reinterpret_cast<uintptr_t>(pooled) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(pooled_bf16) % 8 == 0 && (d / 1024 & (d / 1024 - 1)) == 0;
    if (!vec) return false;
    if (n_req <= 0) return true;
    const int V = d / 1024;   // d = 1024 V: NT = 256 V threads of one float4 up to d = 4096, then 2 each
#define OUTLETS_NPS_V(TY, TG, VV, NT, PER)                                                                 \
    case VV:                                                                                               \
        if (rs)                                                                                            \
            hipLaunchKernelGGL((norm_pool_step_kernel<TY, TG, NT, PER, true>), dim3(n_req), dim3(NT), 0, st, d, \
                               n_req, x, ldx, static_cast<const TG*>(gamma), eps, static_cast<TY*>(y), ldy, y2, \
                               ldy2, req_slot, req_start, pool_sum, pooled, pooled_bf16, *rs);            \
        else                                                                                               \
            hipLaunchKernelGGL((norm_pool_step_kernel<TY, TG, NT, PER>), dim3(n_req), dim3(NT), 0, st, d, n_req, \
                               x, ldx, static_cast<const TG*>(gamma), eps, static_cast<TY*>(y), ldy, y2, ldy2, \
                               req_slot, req_start, pool_sum, pooled, pooled_bf16);                      \
        break;
#define OUTLETS_NPS(TY, TG)                                                                                \
    switch (V) { OUTLETS_NPS_V(TY, TG, 1, 256, 1) OUTLETS_NPS_V(TY, TG, 2, 512, 1)                          \
                 OUTLETS_NPS_V(TY, TG, 4, 1024, 1) OUTLETS_NPS_V(TY, TG, 8, 1024, 2) }
    if (act_fmt == FMT_F32) { OUTLETS_NPS(float, float) }
    else if (gamma_fmt == FMT_F32) { OUTLETS_NPS(bf16_t, float) }
    else { OUTLETS_NPS(bf16_t, bf16_t) }
#undef OUTLETS_NPS
#undef OUTLETS_NPS_V
    return true;
}

void launch_pool_step(int n_req, int d, int h_fmt, const void* h, int64_t ldh, const int32_t* req_slot,
                      const int32_t* req_start, float* pool_sum, float* pooled,
                      uint16_t* pooled_bf16, hipStream_t st) {
    if (n_req <= 0) return;
    const dim3 g(n_req, (d + 255) / 256);
    if (h_fmt == FMT_F32)
        hipLaunchKernelGGL(pool_step_kernel<float>, g, dim3(256), 0, st, d, static_cast<const float*>(h), ldh,
                           req_slot, req_start, pool_sum, pooled, pooled_bf16);
    else
        hipLaunchKernelGGL(pool_step_kernel<bf16_t>, g, dim3(256), 0, st, d, static_cast<const bf16_t*>(h), ldh,
                           req_slot, req_start, pool_sum, pooled, pooled_bf16);
}

namespace {

// Draft model head softmax (Eq. 2): one 1024-thread block per request over
// its V logits; with two_rows the logits are the sum of row i (bf16 hi part
// of the draft state) and row n + i (lo part).
// Softmax over the draft model head's logits, request i's logits being row i
// (plus row n + i, the lo half of the bf16 hi/lo input split).  Each request's
// v logits are cut into kLmChunks chunks, one 256-thread block each: stage 1
// writes each chunk's max and sum of exp(x - max); stage 2 combines the
// request's chunk statistics in chunk order (every block the same way, so the
// result is deterministic) and writes the probabilities of its chunk.  (One
// block per request kept 32 CUs busy: 135 us for 32 requests over 128,256
// logits, against 179 us for the head's 1 GB weight stream.)
constexpr int kLmChunks = 32;

__device__ __forceinline__ void lm_chunk(int v, int c, int& j0, int& j1) {
    const int per = (v + kLmChunks - 1) / kLmChunks;
    j0 = min(v, c * per);
    j1 = min(v, j0 + per);
}

__global__ void __launch_bounds__(256)
lm_softmax_stats_kernel(int n, int v, const float* __restrict__ logits, int two_rows, float* __restrict__ stats) {
    __shared__ float red[4];
    const int i = blockIdx.x, c = blockIdx.y;
    const float* hi = logits + (int64_t)i * v;
    const float* lo = logits + (int64_t)(n + i) * v;
    int j0, j1;
    lm_chunk(v, c, j0, j1);
    float mx = -INFINITY;
    for (int j = j0 + threadIdx.x; j < j1; j += 256) mx = fmaxf(mx, two_rows ? hi[j] + lo[j] : hi[j]);
    mx = wave_max(mx);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    __syncthreads();
    float sum = 0.f;
    if (mx > -INFINITY)
        for (int j = j0 + threadIdx.x; j < j1; j += 256) sum += __expf((two_rows ? hi[j] + lo[j] : hi[j]) - mx);
    sum = block_sum<256>(sum, red);
    if (threadIdx.x == 0) {
        stats[((int64_t)i * kLmChunks + c) * 2] = mx;
        stats[((int64_t)i * kLmChunks + c) * 2 + 1] = sum;
    }
}

__global__ void __launch_bounds__(256)
lm_softmax_norm_kernel(int n, int v, const float* __restrict__ logits, int two_rows,
                       const float* __restrict__ stats, float* __restrict__ p) {
    const int i = blockIdx.x, c = blockIdx.y;
    const float* st = stats + (int64_t)i * kLmChunks * 2;
    float M = -INFINITY;
#pragma unroll
    for (int k = 0; k < kLmChunks; ++k) M = fmaxf(M, st[2 * k]);
    float S = 0.f;
#pragma unroll
    for (int k = 0; k < kLmChunks; ++k)
        if (st[2 * k] > -INFINITY) S += st[2 * k + 1] * __expf(st[2 * k] - M);
    const float inv = 1.0f / S;
    const float* hi = logits + (int64_t)i * v;
    const float* lo = logits + (int64_t)(n + i) * v;
    float* pr = p + (int64_t)i * v;
    int j0, j1;
    lm_chunk(v, c, j0, j1);
    for (int j = j0 + threadIdx.x; j < j1; j += 256) pr[j] = __expf((two_rows ? hi[j] + lo[j] : hi[j]) - M) * inv;
}

}  // namespace

int lm_softmax_stats_floats(int n) { return 2 * kLmChunks * n; }

void launch_lm_softmax(int n, int v, const float* logits, bool two_rows, float* stats, float* p, hipStream_t st) {
    if (n <= 0 || v <= 0) return;
    const dim3 grid(n, kLmChunks);
    hipLaunchKernelGGL(lm_softmax_stats_kernel, grid, dim3(256), 0, st, n, v, logits, two_rows ? 1 : 0, stats);
    hipLaunchKernelGGL(lm_softmax_norm_kernel, grid, dim3(256), 0, st, n, v, logits, two_rows ? 1 : 0, stats, p);
}

void launch_head_finish(int w_fmt, int n_req, int h1, int splits, const float* partial,
                        const void* b1, const void* w2, const void* b2, float* z, hipStream_t st) {
    if (n_req <= 0) return;
    if (splits % 8 == 0 && h1 % 4 == 0) {
        if (w_fmt == FMT_F32)
            hipLaunchKernelGGL((head_finish_vec_kernel<float, 8>), dim3(n_req), dim3(256), 0, st, h1, n_req,
                               n_req, splits, partial, static_cast<const float*>(b1), static_cast<const float*>(w2),
                               static_cast<const float*>(b2), z);
        else
            hipLaunchKernelGGL((head_finish_vec_kernel<bf16_t, 8>), dim3(n_req), dim3(256), 0, st, h1, n_req,
                               2 * n_req, splits, partial, static_cast<const bf16_t*>(b1),
                               static_cast<const bf16_t*>(w2), static_cast<const bf16_t*>(b2), z);
        return;
    }
    if (w_fmt == FMT_F32)
        hipLaunchKernelGGL((head_finish_kernel<float>), dim3(n_req), dim3(256), 0, st, h1, splits,
                           n_req, n_req, partial, static_cast<const float*>(b1),
                           static_cast<const float*>(w2), static_cast<const float*>(b2), z);
    else
        hipLaunchKernelGGL((head_finish_kernel<bf16_t>), dim3(n_req), dim3(256), 0, st, h1, splits,
                           n_req, 2 * n_req, partial, static_cast<const bf16_t*>(b1),
                           static_cast<const bf16_t*>(w2), static_cast<const bf16_t*>(b2), z);
}

void launch_copy_rows_act(int act_fmt, int rows, int d, const float* src, int64_t lds, void* dst,
                          int64_t ldd, hipStream_t st) {
    if (rows <= 0) return;
    if (act_fmt == FMT_F32)
        hipLaunchKernelGGL((copy_rows_kernel<float>), dim3(rows), dim3(256), 0, st, d, src, lds,
                           static_cast<float*>(dst), ldd);
    else
        hipLaunchKernelGGL((copy_rows_kernel<bf16_t>), dim3(rows), dim3(256), 0, st, d, src, lds,
                           static_cast<bf16_t*>(dst), ldd);
}

}  // namespace outlets
