// Attention of the draft decoder layer over the paged draft KV cache.
//
// One workgroup (4 waves) per (query token, KV head): the G = n_q / n_kv
// query heads of the group share every K/V page the workgroup reads.  Keys
// 0..pos of the token's slot are visited page by page (16 keys, hd-contiguous
// rows); page i goes to wave i % 4.  Each wave keeps an online softmax per
// query head (running max m, normaliser l, unnormalised output o) in base 2:
// q is pre-scaled by log2(e) / sqrt(hd) so exp2 gives exp(q.k / sqrt(hd)).
// The four wave states are merged through LDS at the end.
//
// Score phase: lane = key (0..15) + 16 * part; each lane dots hd/4 channels
// and two xor-shuffles complete the dot product.  Value phase: each lane owns
// hd/64 output channels and reads them for all 16 keys of the page.
#include "common.hpp"
#include "kernels.hpp"
#include "outlets.h"

namespace outlets {

namespace {

template <typename T, int HD, int G>
__global__ void __launch_bounds__(256)
attn_paged_kernel(const T* q, int64_t ldq, T* out, int64_t ldo, const int32_t* tok_slot,
                  const int32_t* tok_pos, const int32_t* page_table, int max_pages,
                  const T* kpool, const T* vpool, int n_kv, float qscale) {
    constexpr int NW = 4, DP = HD / 4, DV = HD / 64;
    __shared__ float qs[G][HD];
    __shared__ float sm[NW][G], sl[NW][G];
    __shared__ float so[NW][G][HD];

    const int64_t t = blockIdx.x;
    const int g = blockIdx.y;
    const int pos = tok_pos[t], slot = tok_slot[t];
    const int nkeys = pos + 1, npages = (nkeys + 15) / 16;
    for (int e = threadIdx.x; e < G * HD; e += 256) {
        const int h = e / HD, c = e % HD;
        qs[h][c] = load_act<T>(q + t * ldq + (int64_t)(g * G + h) * HD + c) * qscale;
    }
    __syncthreads();

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int key = lane & 15, part = lane >> 4;
    float m[G], l[G], o[G][DV];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        m[h] = -INFINITY;
        l[h] = 0.f;
#pragma unroll
        for (int d = 0; d < DV; ++d) o[h][d] = 0.f;
    }

    const int32_t* prow = page_table + (int64_t)slot * max_pages;
    for (int pi = w; pi < npages; pi += NW) {
        const int64_t page = prow[pi];
        const T* kb = kpool + (page * n_kv + g) * 16 * HD;
        const T* vb = vpool + (page * n_kv + g) * 16 * HD;
        float kv[DP];
#pragma unroll
        for (int d = 0; d < DP; ++d) kv[d] = load_act<T>(kb + key * HD + part * DP + d);
        // rows past the last key hold stale or never-written data: zero them
        // so the p = 0 weights cannot meet a NaN pattern
        float vv[16][DV];
#pragma unroll
        for (int k = 0; k < 16; ++k)
#pragma unroll
            for (int d = 0; d < DV; ++d)
                vv[k][d] = (pi * 16 + k < nkeys) ? load_act<T>(vb + k * HD + lane * DV + d) : 0.f;
        const bool valid = pi * 16 + key < nkeys;
#pragma unroll
        for (int h = 0; h < G; ++h) {
            float s = 0.f;
#pragma unroll
            for (int d = 0; d < DP; ++d) s = fmaf(qs[h][part * DP + d], kv[d], s);
            s += __shfl_xor(s, 16, 64);
            s += __shfl_xor(s, 32, 64);
            s = valid ? s : -INFINITY;
            float mx = s;
#pragma unroll
            for (int x = 1; x < 16; x <<= 1) mx = fmaxf(mx, __shfl_xor(mx, x, 64));
            const float mn = fmaxf(m[h], mx);   // finite: key 0 of the page is valid
            const float corr = exp2f(m[h] - mn);
            const float p = valid ? exp2f(s - mn) : 0.f;
            float ps = p;
#pragma unroll
            for (int x = 1; x < 16; x <<= 1) ps += __shfl_xor(ps, x, 64);
            l[h] = l[h] * corr + ps;
#pragma unroll
            for (int d = 0; d < DV; ++d) o[h][d] *= corr;
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                const float pk = __shfl(p, k, 64);
#pragma unroll
                for (int d = 0; d < DV; ++d) o[h][d] = fmaf(pk, vv[k][d], o[h][d]);
            }
            m[h] = mn;
        }
    }

    if (lane == 0)
#pragma unroll
        for (int h = 0; h < G; ++h) { sm[w][h] = m[h]; sl[w][h] = l[h]; }
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
        for (int d = 0; d < DV; ++d) so[w][h][lane * DV + d] = o[h][d];
    __syncthreads();
    for (int e = threadIdx.x; e < G * HD; e += 256) {
        const int h = e / HD, c = e % HD;
        float mx = -INFINITY;
#pragma unroll
        for (int v = 0; v < NW; ++v) mx = fmaxf(mx, sm[v][h]);
        float L = 0.f, O = 0.f;
#pragma unroll
        for (int v = 0; v < NW; ++v) {
            if (sm[v][h] == -INFINITY) continue;   // wave had no page
            const float f = exp2f(sm[v][h] - mx);
            L = fmaf(sl[v][h], f, L);
            O = fmaf(so[v][h][c], f, O);
        }
        store_act<T>(out + t * ldo + (int64_t)(g * G + h) * HD + c, O / L);
    }
}

template <typename T, int HD>
bool launch_hd(int G, int ntok, const void* q, int64_t ldq, void* out, int64_t ldo,
               const int32_t* tok_slot, const int32_t* tok_pos, const int32_t* page_table,
               int max_pages, const void* kpool, const void* vpool, int n_kv, float qscale,
               hipStream_t st) {
    dim3 grid(ntok, n_kv);
#define OUTLETS_ATTN_G(GG)                                                                     \
    case GG:                                                                                   \
        hipLaunchKernelGGL((attn_paged_kernel<T, HD, GG>), grid, dim3(256), 0, st,             \
                           static_cast<const T*>(q), ldq, static_cast<T*>(out), ldo, tok_slot,  \
                           tok_pos, page_table, max_pages, static_cast<const T*>(kpool),       \
                           static_cast<const T*>(vpool), n_kv, qscale);                        \
        return true;
    switch (G) {
        OUTLETS_ATTN_G(1)
        OUTLETS_ATTN_G(2)
        OUTLETS_ATTN_G(4)
        OUTLETS_ATTN_G(8)
    }
#undef OUTLETS_ATTN_G
    return false;
}

}  // namespace

bool attn_supported(int n_q, int n_kv, int hd) {
    if (n_kv <= 0 || n_q % n_kv) return false;
    const int G = n_q / n_kv;
    return (G == 1 || G == 2 || G == 4 || G == 8) && (hd == 64 || hd == 128);
}

void launch_attn_paged(int act_fmt, int ntok, const void* q, int64_t ldq, void* out,
                       int64_t ldo, const int32_t* tok_slot, const int32_t* tok_pos,
                       const int32_t* page_table, int max_pages, const void* kpool,
                       const void* vpool, int n_q, int n_kv, int hd, hipStream_t st) {
    if (ntok <= 0) return;
    const int G = n_q / n_kv;
    const float qscale = 1.4426950408889634f / sqrtf(static_cast<float>(hd));
    if (act_fmt == FMT_F32) {
        if (hd == 64) launch_hd<float, 64>(G, ntok, q, ldq, out, ldo, tok_slot, tok_pos, page_table, max_pages, kpool, vpool, n_kv, qscale, st);
        else launch_hd<float, 128>(G, ntok, q, ldq, out, ldo, tok_slot, tok_pos, page_table, max_pages, kpool, vpool, n_kv, qscale, st);
    } else {
        if (hd == 64) launch_hd<bf16_t, 64>(G, ntok, q, ldq, out, ldo, tok_slot, tok_pos, page_table, max_pages, kpool, vpool, n_kv, qscale, st);
        else launch_hd<bf16_t, 128>(G, ntok, q, ldq, out, ldo, tok_slot, tok_pos, page_table, max_pages, kpool, vpool, n_kv, qscale, st);
    }
}

}  // namespace outlets
