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
// hd/64 output channels and reads them for all 16 keys of the page (value
// pages are stored [hd][16 tokens]).
//
// Prefill (bf16, hd 128): a flash-attention kernel on MFMA, see below.
#include <type_traits>

#include <algorithm>
#include <vector>

#include "common.hpp"
#include "kernels.hpp"
#include "outlets.h"

namespace outlets {

namespace {

// 2^x with the hardware v_exp_f32 (results below 2^-126 flush to zero, which
// only ever drops probabilities that vanish next to the running maximum).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Gated Attention output gate: sigmoid of the gate projection (gate values
// sit in the q|k|v|g row, one per query-head channel).
__device__ __forceinline__ float sigmoid_f(float x) {
    return __builtin_amdgcn_rcpf(1.0f + fast_exp2(-1.4426950408889634f * x));
}

// 16-byte LDS DMA per lane (lane i writes lds_base + 16 i), its wait, and a
// workgroup barrier without the release fence (the DMA is ordered by the
// explicit wait; the empty asm statements keep the compiler from moving
// memory accesses across the barrier).
__device__ __forceinline__ void dma_16(const void* g, char* lds_base) {
    __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds_base, 16, 0, 0);
}
__device__ __forceinline__ void wait_vm0() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void block_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <typename T, int HD, int G>
__global__ void __launch_bounds__(256)
attn_paged_kernel(const T* q, int64_t ldq, T* out, int64_t ldo, const int32_t* tok_slot,
                  const int32_t* tok_pos, const int32_t* page_table, int max_pages,
                  const T* kpool, const T* vpool, int n_kv, float qscale, const T* gate) {
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
                vv[k][d] = (pi * 16 + k < nkeys) ? load_act<T>(vb + (lane * DV + d) * 16 + k) : 0.f;
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
            const float corr = fast_exp2(m[h] - mn);
            const float p = valid ? fast_exp2(s - mn) : 0.f;
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
            const float f = fast_exp2(sm[v][h] - mx);
            L = fmaf(sl[v][h], f, L);
            O = fmaf(so[v][h][c], f, O);
        }
        float y = O / L;
        if (gate) y *= sigmoid_f(load_act<T>(gate + t * ldq + (int64_t)(g * G + h) * HD + c));
        store_act<T>(out + t * ldo + (int64_t)(g * G + h) * HD + c, y);
    }
}

// ---------------------------------------------------------------- prefill, MFMA
// Query blocks per wave (32 queries each).  One block keeps a wave within
// 256 registers, so two waves share each SIMD and one's softmax overlaps the
// other's MFMAs; this measured faster than two blocks per wave (which share
// every K/V fragment read but need 400+ registers, one wave per SIMD).
#ifndef OUTLETS_PREFILL_QB
#define OUTLETS_PREFILL_QB 1   // query blocks per wave for 2 and 4 heads per group
#endif
constexpr int prefill_blocks(int G) { return (G == 2 || G == 4) ? OUTLETS_PREFILL_QB : 1; }


// One workgroup per (request, tile of 32 QB WB queries, KV head); wave w
// computes query head g * G + w % G for its QB blocks of 32 queries (block
// w / G of the WB the workgroup holds), so the G heads of a group and the WB
// blocks share each K/V tile, and a wave's blocks share every fragment read
// from LDS.  Keys are visited in tiles of 64 (4 pages) up to the tile's last query
// position (causal tile skipping); tiles are copied into two LDS stages by
// DMA while the previous tile is multiplied.
//
// Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16:
// a lane then holds one query (column) and 16 keys per 32x32 block, so the
// online softmax max/sum need one cross-half shuffle and the rescaling of the
// output is lane-local.  The output is also kept transposed, O^T = V^T P^T,
// which takes P straight from the score registers as the B operand.  For the
// 8 key values a lane half supplies to one MFMA to be contiguous keys, A row
// rho of the score MFMA reads key pi(rho), pi swapping bits 2 and 3 of rho:
// with the 32x32 output layout (row = 8 (r / 4) + 4 half + r % 4 for
// accumulator element r) element r then holds key 16 (r / 8) + 8 half + r % 8.
// Values are staged as the tile's four transposed value pages, [page][hd][16
// keys], each a plain copy of its page block.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two workgroups per CU for one 32-query block per wave and at least four
// waves (the benchmark shapes, G = 4 and 8); the one- and two-wave groups of
// G = 1 and 2 (reduced test shapes) need more than half a SIMD's registers,
// so they ask for one.
template <int G, int QB, int WB>
__global__ void __launch_bounds__(G * WB * 64, (QB == 1 && G >= 4) ? 2 : 1)
attn_prefill_mfma(const bf16_t* qkv, int64_t ldq, bf16_t* out, int64_t ldo, const int32_t* work,
                  const int32_t* req_off, const int32_t* req_slot, const int32_t* page_table,
                  int max_pages, const bf16_t* kpool, const bf16_t* vpool, int n_kv, float qscale,
                  const bf16_t* gate) {
    constexpr int HD = 128, NW = G * WB, BKV = 64, NS = HD / 16, NB = HD / 32, QT = 32 * QB * WB;
    constexpr int KB = BKV * HD * 2, STAGE = 2 * KB;    // K [64][128] + V^T [128][64], bf16
    constexpr int KCP = (KB / 1024) / NW;               // DMA copies per wave for K (and for V)
    __shared__ __attribute__((aligned(16))) char lds[2 * STAGE];

    const int r = work[2 * blockIdx.x], qt = work[2 * blockIdx.x + 1];
    const int g = blockIdx.y;
    const int tok0 = req_off[r], n = req_off[r + 1] - tok0, slot = req_slot[r];
    const int qs = qt * QT;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int l32 = lane & 31, hf = lane >> 5;
    const int h = g * G + w % G;
    const int qsw = qs + 32 * QB * (w / G);   // this wave's first query
    const int32_t* prow = page_table + (int64_t)slot * max_pages;
    const int last_page = (n - 1) >> 4;

    // queries of this lane: block qb covers positions qs + 32 qb + l32 (tail lanes repeat the last)
    int tp[QB];
    bf16x8 qf[QB][NS];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        tp[qb] = min(qsw + 32 * qb + l32, n - 1);
        const bf16_t* qrow = qkv + (int64_t)(tok0 + tp[qb]) * ldq + h * HD + hf * 8;
#pragma unroll
        for (int s2 = 0; s2 < NS; ++s2)
            qf[qb][s2] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(qrow + 16 * s2));
    }
    f32x16 o[QB][NB];
    float m[QB], lsum[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        m[qb] = -INFINITY;
        lsum[qb] = 0.f;
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e) o[qb][b][e] = 0.f;
    }
    const int maxpos = min(qs + QT - 1, n - 1);
    const int ntiles = maxpos / BKV + 1;
    const int arow_key = (l32 & 19) | ((l32 & 4) << 1) | ((l32 & 8) >> 1);

    // DMA of one 64-key tile: K rows (key, 16 chunks of 8 channels, chunk c at
    // c ^ key%16) and the four V^T page blocks as they are in the pool.  Copy
    // cp (1 KiB) is K keys 4 cp .. 4 cp + 3 and V channels 32 (cp % 4) ..
    // +31 of the tile's page cp / 4, so every copy reads one page: its id is
    // uniform (read-first-lane) and the address is a scalar base plus a
    // 32-bit lane offset.  Page ids are loaded one tile ahead; pages past the
    // prompt's last one repeat it.  Keys past the prompt are masked out of
    // the scores and their (finite) rows get weight 0.
    const int wu = __builtin_amdgcn_readfirstlane(w);
    // this wave's copies cover PPW pages of a tile, starting at page q0
    constexpr int PPW = KCP >= 4 ? KCP / 4 : 1;
    const int q0 = (wu * KCP) >> 2;
    auto load_pages = [&](int kt, int* pg) {
#pragma unroll
        for (int i = 0; i < PPW; ++i) pg[i] = prow[min(4 * kt + q0 + i, last_page)];
    };
    auto issue = [&](const int* pgv, int stage) {
        char* base = lds + stage * STAGE;
        int ps[PPW];
#pragma unroll
        for (int i = 0; i < PPW; ++i) ps[i] = __builtin_amdgcn_readfirstlane(pgv[i]);
#pragma unroll
        for (int j = 0; j < KCP; ++j) {
            const int cp = wu * KCP + j;
            const int page = ps[KCP >= 4 ? j >> 2 : 0];
            const int key = (cp & 3) * 4 + (lane >> 4);          // key within the page
            const int c = (lane & 15) ^ key;
            const bf16_t* src = kpool + ((int64_t)page * n_kv + g) * (16 * HD);
            dma_16(src + (key * HD + c * 8), base + cp * 1024);
        }
#pragma unroll
        for (int j = 0; j < KCP; ++j) {
            const int cp = wu * KCP + j;
            const int page = ps[KCP >= 4 ? j >> 2 : 0];
            const bf16_t* src = vpool + ((int64_t)page * n_kv + g) * (HD * 16);
            dma_16(src + ((cp & 3) * 512 + lane * 8), base + KB + cp * 1024);
        }
    };

    int pgn[PPW];   // this wave's page ids of the next tile to copy

    // One 64-key tile.  MASKED: apply the causal mask (tiles holding a key
    // past the tile's first query); tiles wholly before it skip the mask.
    // The running max m is kept pre-scaled (log2 units), so one FMA forms the
    // exponent of each probability.
    auto tile = [&](int kt, auto masked_tag) {
        constexpr bool MASKED = decltype(masked_tag)::value;
        wait_vm0();
        block_barrier();      // tile kt is in LDS; every wave is done with tile kt-1
        issue(pgn, (kt + 1) & 1);                       // tile min(kt + 1, ntiles - 1)
        load_pages(min(kt + 2, ntiles - 1), pgn);
        const char* ks = lds + (kt & 1) * STAGE;
        const char* vs = ks + KB;
        const int k0 = kt * BKV;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            f32x16 sacc[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int e = 0; e < 16; ++e) sacc[kb][e] = 0.f;
                const int key = 32 * kb + arow_key;
#pragma unroll
                for (int s2 = 0; s2 < NS; ++s2) {
                    const int ch = 2 * s2 + hf;
                    const bf16x8 a = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(ks + key * 256 + ((ch ^ (key & 15)) << 4)));
                    sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[qb][s2], sacc[kb], 0, 0, 0);
                }
            }
            // interleave the K fragment reads with the score MFMAs (left to
            // itself the scheduler read two fragments, waited, and issued one
            // MFMA; measured on the 32-request 8B batch: 0.607-0.627 ->
            // 0.583-0.589 ms)
            __builtin_amdgcn_iglp_opt(1);
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    if (MASKED) {
                        const int kpos = k0 + 32 * kb + 16 * (e >> 3) + 8 * hf + (e & 7);
                        if (kpos > tp[qb]) sacc[kb][e] = -INFINITY;
                    }
                    mx = fmaxf(mx, sacc[kb][e]);
                }
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * qscale;   // finite: key 0 <= every query position
            // The reference max m moves only when the tile's max exceeds it by
            // more than 8 (probabilities then stay <= 2^8), so the rescaling of
            // O and l is skipped, wave-uniformly, on most tiles; O / l is
            // unchanged by the choice of reference.
            const bool grow = mx > m[qb] + 8.f;
            if (__any(grow)) {
                const float mn = grow ? mx : m[qb];
                const float corr = fast_exp2(m[qb] - mn);
                m[qb] = mn;
                lsum[qb] *= corr;
#pragma unroll
                for (int b = 0; b < NB; ++b)
#pragma unroll
                    for (int e = 0; e < 16; ++e) o[qb][b][e] *= corr;
            }
            const float nmn = -m[qb];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int e = 0; e < 16; ++e) sacc[kb][e] = fast_exp2(fmaf(sacc[kb][e], qscale, nmn));
            // The probabilities enter the PV product as bf16; the row sum adds
            // the same bf16 values, two per dot2 instruction, so the output is
            // a convex combination of the value rows.
            bf16x8 pbs[2][2];
            float ps = 0.f;
            const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int u = 0; u < 2; ++u) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) pbs[kb][u][e] = static_cast<__bf16>(sacc[kb][8 * u + e]);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const bf16x2 pr = {pbs[kb][u][2 * e], pbs[kb][u][2 * e + 1]};
                        ps = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, ps, false);
                    }
                }
            lsum[qb] += ps + __shfl_xor(ps, 32, 64);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const bf16x8 pb = pbs[kb][u];
                    const int ch = 4 * kb + 2 * u + hf;
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        const int row = 32 * b + l32;
                        const bf16x8 a = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(vs + (ch >> 1) * 4096 + row * 32 + (ch & 1) * 16));
                        o[qb][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, o[qb][b], 0, 0, 0);
                    }
                }
            __builtin_amdgcn_iglp_opt(1);   // the same for the V fragments and the PV MFMAs
        }
    };

    load_pages(0, pgn);
    issue(pgn, 0);
    load_pages(min(1, ntiles - 1), pgn);
    // tiles whose last key (64 kt + 63) is at or before this wave's first query
    const int nfull = min(ntiles, (qsw + 1) / BKV);
    for (int kt = 0; kt < nfull; ++kt) tile(kt, std::false_type{});
    for (int kt = nfull; kt < ntiles; ++kt) tile(kt, std::true_type{});
    wait_vm0();   // the last (duplicate) tile copy must land before the workgroup ends
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int q = qsw + 32 * qb + l32;
        if (q >= n) continue;
        bf16_t* orow = out + (int64_t)(tok0 + q) * ldo + h * HD;
        const float inv = 1.0f / lsum[qb];
        const bf16_t* grow = gate ? gate + (int64_t)(tok0 + q) * ldq + h * HD : nullptr;
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int c0 = 32 * b + 8 * j + 4 * hf;
                float y[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) y[e] = o[qb][b][4 * j + e] * inv;
                if (grow) {
                    const uint2 gv = *reinterpret_cast<const uint2*>(grow + c0);
                    y[0] *= sigmoid_f(__uint_as_float(gv.x << 16));
                    y[1] *= sigmoid_f(__uint_as_float(gv.x & 0xffff0000u));
                    y[2] *= sigmoid_f(__uint_as_float(gv.y << 16));
                    y[3] *= sigmoid_f(__uint_as_float(gv.y & 0xffff0000u));
                }
                uint2 pk;
                pk.x = f32_to_bf16(y[0]) | (uint32_t(f32_to_bf16(y[1])) << 16);
                pk.y = f32_to_bf16(y[2]) | (uint32_t(f32_to_bf16(y[3])) << 16);
                *reinterpret_cast<uint2*>(orow + c0) = pk;
            }
    }
}

// ---------------------------------------------------------------- decode, MFMA
// One query token per request (a decode step).  Split-KV over contiguous page
// ranges: the step's pages, requests in order, are cut into equal ranges, one
// per wave and KV head (attn_decode_plan).  A wave's range splits at request
// ends into segments; each segment keeps one online softmax for the G query
// heads of the KV head and leaves one (m, l, o) partial record, which
// attn_decode_combine merges in segment order (deterministic).  Segments are
// walked in pieces of at most kDecodeChunk pages (one page id per lane).
//
// Per 16-key page: S = K Q^T with v_mfma_f32_16x16x32_bf16 (A = K rows, lane
// l -> key l % 16; B = Q^T with the G heads in columns 0..G-1 of 16, the rest
// zero); the 16x16 output gives lane l the scores of head l % 16 for keys
// 4 (l / 16) + i, which is exactly the B-operand layout of
// O^T += V^T P^T with v_mfma_f32_16x16x16bf16_1k (A = V^T rows from the
// transposed value page).  The softmax is lane-local plus two xor-shuffles.
// The next pages' K/V fragments are loaded before the current ones are used.
#ifndef OUTLETS_DECODE_CHUNK
#define OUTLETS_DECODE_CHUNK 64
#endif
#ifndef OUTLETS_DECODE_PPI
#define OUTLETS_DECODE_PPI 2
#endif
constexpr int kDecodeChunk = OUTLETS_DECODE_CHUNK;
constexpr int kDecodeRec = 128 + 4;   // floats per partial record: m, l, 2 pad, o[128]

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <int G>
__global__ void __launch_bounds__(64)
attn_decode_mfma(const bf16_t* __restrict__ q, int64_t ldq, const int32_t* __restrict__ work,
                 const int32_t* __restrict__ lanes, const int32_t* __restrict__ req_slot,
                 const int32_t* __restrict__ req_start, const int32_t* __restrict__ page_table, int max_pages,
                 const bf16_t* __restrict__ kpool, const bf16_t* __restrict__ vpool, int n_kv, float qscale,
                 float* __restrict__ part) {
    constexpr int HD = 128;
    static_assert(G <= 16, "query heads per KV head");
    static_assert(kDecodeChunk <= 64, "one page id per lane");
    const int g = blockIdx.y;
    const int lane = threadIdx.x, col = lane & 15, grp = lane >> 4;
    const int j0 = lanes[blockIdx.x], j1 = lanes[blockIdx.x + 1];   // this wave's pieces

    // Partial records are staged in LDS and stored with full-wave 16-byte
    // non-temporal stores after the next piece's first page loads are
    // issued.  Storing them straight from the accumulators (nine partial-wave
    // stores, whose registers the next piece overwrites at once) stalled the
    // wave behind the saturated read stream: measured 1.52 against 1.455 ms
    // for the attention of a 512-request step over 2.19M cached tokens.
    __shared__ __attribute__((aligned(16))) float stage[G * kDecodeRec];
    constexpr int RCH = G * kDecodeRec / 4;             // 16-byte chunks of a record block
    int staged = -1;                                    // segment whose record sits in `stage`
    auto flush = [&]() {
        const f32x4* src = reinterpret_cast<const f32x4*>(stage);
        f32x4* dst = reinterpret_cast<f32x4*>(part + ((int64_t)staged * n_kv + g) * G * kDecodeRec);
#pragma unroll
        for (int k = 0; k < (RCH + 63) / 64; ++k) {
            const int ch = lane + 64 * k;
            if (ch < RCH) __builtin_nontemporal_store(src[ch], dst + ch);
        }
        staged = -1;
    };

    float m = -INFINITY, l = 0.f;
    f32x4 o[HD / 16];
    int seg = -1;
    for (int j = j0; j < j1; ++j) {
        const int r = work[4 * j], p0 = work[4 * j + 1], p1 = work[4 * j + 2];
        if (work[4 * j + 3] != seg) {                   // a new segment: fresh softmax state
            seg = work[4 * j + 3];
            m = -INFINITY;
            l = 0.f;
#pragma unroll
            for (int cb = 0; cb < HD / 16; ++cb) o[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        const int slot = req_slot[r];
        const int nkeys = req_start[r] + 1;            // cached keys plus the new token's

        bf16x8 qb[HD / 32];
        {
            const bf16_t* qrow = q + (int64_t)r * ldq + (int64_t)(g * G + min(col, G - 1)) * HD + 8 * grp;
#pragma unroll
            for (int b = 0; b < HD / 32; ++b) {
                uint4 v = *reinterpret_cast<const uint4*>(qrow + 32 * b);
                if (col >= G) v = make_uint4(0u, 0u, 0u, 0u);
                qb[b] = __builtin_bit_cast(bf16x8, v);
            }
        }

        // the piece's page ids, one per lane, fetched up front so the K/V loads of
        // a page never wait on its page-table entry
        const int32_t* prow = page_table + (int64_t)slot * max_pages;
        const int my_page = (p0 + lane < p1) ? prow[p0 + lane] : 0;
        // PPI pages per iteration: their K/V fragments for the next iteration are
        // loaded before this iteration's pages are used (2 * PPI pages in flight)
        constexpr int PPI = OUTLETS_DECODE_PPI;
        uint4 kc[PPI][HD / 32], kn[PPI][HD / 32];
        uint2 vc[PPI][HD / 16], vn[PPI][HD / 16];
        // K/V pages are read once per step: non-temporal loads (measured on this
        // access pattern, loads alone: 6.6 TB/s against 5.9 TB/s with ordinary
        // loads, which a plain sequential read of the pools does not beat)
        auto load_page = [&](int pi, uint4* kf, uint2* vf) {
            const int64_t page = __shfl(my_page, min(pi, p1 - 1) - p0, 64);
            const bf16_t* kb = kpool + (page * n_kv + g) * 16 * HD + col * HD + 8 * grp;
            const bf16_t* vb = vpool + (page * n_kv + g) * HD * 16 + col * 16 + 4 * grp;
#pragma unroll
            for (int b = 0; b < HD / 32; ++b)
                kf[b] = __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kb + 32 * b)));
#pragma unroll
            for (int cb = 0; cb < HD / 16; ++cb)
                vf[cb] = __builtin_bit_cast(uint2, __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(vb + 16 * 16 * cb)));
        };
        auto one_page = [&](int pi, const uint4* kf, const uint2* vf) {
            f32x4 sc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int b = 0; b < HD / 32; ++b)
                sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kf[b]), qb[b], sc, 0, 0, 0);
            // lane: head col, keys 4 grp + i of this page; only the request's last
            // page holds keys past the end (wave-uniform)
            const int k0 = pi * 16 + 4 * grp;
            const bool last = pi * 16 + 16 > nkeys;
            if (last) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (k0 + i >= nkeys) sc[i] = -INFINITY;
            }
            float mx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
            mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            mx *= qscale;                                   // finite: key 16 pi < nkeys
            // The reference max m moves only when the page's max exceeds it by
            // more than 8 (probabilities then stay <= 2^8), so the rescaling of o
            // and l is skipped, wave-uniformly, on most pages; o / l and the
            // merge of the partial records do not depend on the reference.
            const bool grow = mx > m + 8.f;
            if (__any(grow)) {
                const float mn = grow ? mx : m;
                const float corr = fast_exp2(m - mn);
                m = mn;
                l *= corr;
#pragma unroll
                for (int cb = 0; cb < HD / 16; ++cb) o[cb] = o[cb] * corr;
            }
            // the probabilities enter the PV product as bf16 and the row sum adds
            // the same bf16 values, so the output is a convex combination of the
            // value rows
            const float nm = -m;
            float ps = 0.f;
            s16x4 pb;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint16_t pv = f32_to_bf16(fast_exp2(fmaf(sc[i], qscale, nm)));
                pb[i] = static_cast<short>(pv);
                ps += bf16_to_f32(pv);
            }
            ps += __shfl_xor(ps, 16, 64);
            ps += __shfl_xor(ps, 32, 64);
            l += ps;
            // value rows of keys past the end may hold stale data: zero them
#pragma unroll
            for (int cb = 0; cb < HD / 16; ++cb) {
                uint2 vv = vf[cb];
                if (last) {
                    if (k0 + 0 >= nkeys) vv.x &= 0xFFFF0000u;
                    if (k0 + 1 >= nkeys) vv.x &= 0x0000FFFFu;
                    if (k0 + 2 >= nkeys) vv.y &= 0xFFFF0000u;
                    if (k0 + 3 >= nkeys) vv.y &= 0x0000FFFFu;
                }
                o[cb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, vv), pb, o[cb], 0, 0, 0);
            }
        };
#pragma unroll
        for (int u = 0; u < PPI; ++u) load_page(p0 + u, kc[u], vc[u]);
        if (staged >= 0) flush();
        for (int pi = p0; pi < p1; pi += PPI) {
            if (pi + PPI < p1) {
#pragma unroll
                for (int u = 0; u < PPI; ++u) load_page(pi + PPI + u, kn[u], vn[u]);
            }
#pragma unroll
            for (int u = 0; u < PPI; ++u)
                if (pi + u < p1) one_page(pi + u, kc[u], vc[u]);
            if (pi + PPI < p1) {
#pragma unroll
                for (int u = 0; u < PPI; ++u) {
#pragma unroll
                    for (int b = 0; b < HD / 32; ++b) kc[u][b] = kn[u][b];
#pragma unroll
                    for (int cb = 0; cb < HD / 16; ++cb) vc[u][cb] = vn[u][cb];
                }
            }
        }
        // at the segment's end, its record [m, l, -, -, o[0..HD)] per query head
        // g G + col (o 16-byte aligned) goes to the staging area
        if (j + 1 == j1 || work[4 * (j + 1) + 3] != seg) {
            if (col < G) {
                float* rec = stage + col * kDecodeRec;
                if (grp == 0) { rec[0] = m; rec[1] = l; }
#pragma unroll
                for (int cb = 0; cb < HD / 16; ++cb) *reinterpret_cast<f32x4*>(rec + 4 + 16 * cb + 4 * grp) = o[cb];
            }
            staged = seg;
        }
    }
    if (staged >= 0) flush();
}

// Merge of a request's segment partials, in segment (page) order
// (deterministic).  Grid (n_req, ceil(n_q / 8)), 256 threads: 32 threads per
// query head, 4 channels each.  The segments' maxima give the common
// reference M; segment c's o and l enter with weight 2^(m_c - M).
__global__ void __launch_bounds__(256)
attn_decode_combine(const int32_t* cu_segs, const float* part, int n_q, bf16_t* out, int64_t ldo,
                    const bf16_t* gate, int64_t ldg) {
    constexpr int HD = 128;
    const int r = blockIdx.x, h = blockIdx.y * 8 + (threadIdx.x >> 5), ch = (threadIdx.x & 31) * 4;
    if (h >= n_q) return;
    const int c0 = cu_segs[r], c1 = cu_segs[r + 1];
    float M = -INFINITY;
    for (int c = c0; c < c1; ++c) M = fmaxf(M, part[((int64_t)c * n_q + h) * kDecodeRec]);
    float L = 0.f;
    f32x4 O = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int c = c0; c < c1; ++c) {
        const float* rec = part + ((int64_t)c * n_q + h) * kDecodeRec;
        const float2 ml = *reinterpret_cast<const float2*>(rec);
        const f32x4 v = *reinterpret_cast<const f32x4*>(rec + 4 + ch);
        const float f = fast_exp2(ml.x - M);
        L = fmaf(ml.y, f, L);
#pragma unroll
        for (int j = 0; j < 4; ++j) O[j] = fmaf(v[j], f, O[j]);
    }
    float y[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) y[j] = O[j] / L;
    const int64_t col0 = (int64_t)h * HD + ch;
    if (gate) {
        const bf16_t* gr = gate + (int64_t)r * ldg + col0;
#pragma unroll
        for (int j = 0; j < 4; ++j) y[j] *= sigmoid_f(bf16_to_f32(gr[j]));
    }
    *reinterpret_cast<uint2*>(out + (int64_t)r * ldo + col0) =
        make_uint2(f32_to_bf16(y[0]) | (uint32_t(f32_to_bf16(y[1])) << 16),
                   f32_to_bf16(y[2]) | (uint32_t(f32_to_bf16(y[3])) << 16));
}

template <typename T, int HD>
bool launch_hd(int G, int ntok, const void* q, int64_t ldq, void* out, int64_t ldo,
               const int32_t* tok_slot, const int32_t* tok_pos, const int32_t* page_table,
               int max_pages, const void* kpool, const void* vpool, int n_kv, float qscale,
               const void* gate, hipStream_t st) {
    dim3 grid(ntok, n_kv);
#define OUTLETS_ATTN_G(GG)                                                                     \
    case GG:                                                                                   \
        hipLaunchKernelGGL((attn_paged_kernel<T, HD, GG>), grid, dim3(256), 0, st,             \
                           static_cast<const T*>(q), ldq, static_cast<T*>(out), ldo, tok_slot,  \
                           tok_pos, page_table, max_pages, static_cast<const T*>(kpool),       \
                           static_cast<const T*>(vpool), n_kv, qscale,                         \
                           static_cast<const T*>(gate));                                       \
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

// 4 heads per group and prompts of 1,024 tokens or more on average: two
// 32-query blocks per workgroup (8 waves share each K/V tile, half the tile
// copies per query; measured on 466k tokens of 1,821 on average: attention
// 18.8 -> 17.3 ms; on 906 on average: 1.5% slower, so shorter prompts keep 32)
int attn_prefill_query_tile(int n_q, int n_kv, int64_t tokens, int n_req) {
    const int G = n_q / n_kv;
    if (G == 4 && prefill_blocks(G) == 1 && n_req > 0 && tokens >= 1024LL * n_req) return 64;
    return 32 * prefill_blocks(G);
}

bool attn_prefill_mfma_supported(int act_fmt, int n_q, int n_kv, int hd) {
    const int G = n_q / n_kv;
    return act_fmt == FMT_BF16 && hd == 128 && (G == 1 || G == 2 || G == 4 || G == 8);
}

void launch_attn_prefill(int n_work, const int32_t* work, int qtile, const void* qkv, int64_t ldq, void* out,
                         int64_t ldo, const int32_t* req_off, const int32_t* req_slot,
                         const int32_t* page_table, int max_pages, const void* kpool,
                         const void* vpool, int n_q, int n_kv, const void* gate, hipStream_t st) {
    if (n_work <= 0) return;
    const int G = n_q / n_kv;
    const float qscale = 1.4426950408889634f / sqrtf(128.0f);
    dim3 grid(n_work, n_kv);
    if (G == 4 && qtile == 64 && prefill_blocks(4) == 1) {
        hipLaunchKernelGGL((attn_prefill_mfma<4, 1, 2>), grid, dim3(512), 0, st, static_cast<const bf16_t*>(qkv), ldq,
                           static_cast<bf16_t*>(out), ldo, work, req_off, req_slot, page_table, max_pages,
                           static_cast<const bf16_t*>(kpool), static_cast<const bf16_t*>(vpool), n_kv, qscale,
                           static_cast<const bf16_t*>(gate));
        return;
    }
#define OUTLETS_PF_G(GG)                                                                        \
    case GG:                                                                                    \
        hipLaunchKernelGGL((attn_prefill_mfma<GG, prefill_blocks(GG), 1>), grid, dim3(GG * 64), 0, st, \
                           static_cast<const bf16_t*>(qkv), ldq, static_cast<bf16_t*>(out), ldo, \
                           work, req_off, req_slot, page_table, max_pages,                      \
                           static_cast<const bf16_t*>(kpool), static_cast<const bf16_t*>(vpool), \
                           n_kv, qscale, static_cast<const bf16_t*>(gate));                     \
        break;
    switch (G) {
        OUTLETS_PF_G(1)
        OUTLETS_PF_G(2)
        OUTLETS_PF_G(4)
        OUTLETS_PF_G(8)
    }
#undef OUTLETS_PF_G
}

int attn_decode_record_floats() { return kDecodeRec; }

// Lists of the decode waves (per KV head): at most two waves per SIMD (the
// kernel's registers allow two), and at least ~16 pages per wave so that the
// per-piece fixed costs stay small next to the page stream.
static int64_t decode_lane_count(int64_t pages, int n_kv, int cus) {
    const int64_t cap = std::max<int64_t>(1, 8LL * cus / std::max(1, n_kv));
    return std::max<int64_t>(1, std::min<int64_t>(cap, (pages + 15) / 16));
}

int64_t attn_decode_max_segments(int64_t max_req, int n_kv, int cus) {
    return max_req + std::max<int64_t>(1, 8LL * cus / std::max(1, n_kv));
}

int64_t attn_decode_max_pieces(int64_t max_req, int64_t max_pages, int n_kv, int cus) {
    return max_req * ((max_pages + kDecodeChunk - 1) / kDecodeChunk) + attn_decode_max_segments(max_req, n_kv, cus);
}

// The step's pages, requests in order, cut into L ranges whose lengths differ
// by at most one page; a range's part in one request is a segment (one
// partial record), walked in pieces of at most kDecodeChunk pages.  Segments
// are numbered in page order, so each request's segments are consecutive and
// in order.  A segment count of at most L + n_req and a piece count of at most
// pages / kDecodeChunk + segments follow.
void attn_decode_plan(int n_req, const int32_t* pages, int n_kv, int cus, DecodePlan* plan) {
    plan->work.clear();
    plan->lanes.clear();
    plan->cu_segs.assign(n_req + 1, 0);
    std::vector<int64_t> cum(n_req + 1, 0);
    for (int i = 0; i < n_req; ++i) cum[i + 1] = cum[i] + pages[i];
    const int64_t P = cum[n_req];
    const int64_t L = decode_lane_count(P, n_kv, cus);
    plan->n_lanes = static_cast<int>(L);
    plan->lanes.reserve(L + 1);
    int r = 0, n_segs = 0;
    for (int64_t ln = 0; ln < L; ++ln) {
        plan->lanes.push_back(static_cast<int32_t>(plan->work.size() / 4));
        int64_t g = P * ln / L;
        const int64_t e = P * (ln + 1) / L;
        while (g < e) {
            while (cum[r + 1] <= g) ++r;                // the request holding global page g
            if (cum[r] == g) plan->cu_segs[r] = n_segs; // its first segment
            const int64_t se = std::min(e, cum[r + 1]);
            for (int64_t p = g - cum[r]; p < se - cum[r]; p += kDecodeChunk) {
                const int64_t pe = std::min<int64_t>(se - cum[r], p + kDecodeChunk);
                plan->work.insert(plan->work.end(), {r, static_cast<int32_t>(p), static_cast<int32_t>(pe), n_segs});
            }
            ++n_segs;
            g = se;
        }
    }
    plan->lanes.push_back(static_cast<int32_t>(plan->work.size() / 4));
    plan->cu_segs[n_req] = n_segs;
    plan->n_segs = n_segs;
}

void launch_attn_decode(int n_req, int n_pieces, const int32_t* work, const int32_t* cu_segs, int n_lanes,
                        const int32_t* lanes, const void* q, int64_t ldq, void* out, int64_t ldo,
                        const int32_t* req_slot, const int32_t* req_start, const int32_t* page_table, int max_pages,
                        const void* kpool, const void* vpool, int n_q, int n_kv, float* part,
                        const void* gate, hipStream_t st) {
    if (n_req <= 0 || n_pieces <= 0 || n_lanes <= 0) return;
    const int G = n_q / n_kv;
    const float qscale = 1.4426950408889634f / sqrtf(128.0f);
#define OUTLETS_DEC_G(GG)                                                                          \
    case GG:                                                                                       \
        hipLaunchKernelGGL((attn_decode_mfma<GG>), dim3(n_lanes, n_kv), dim3(64), 0, st,           \
                           static_cast<const bf16_t*>(q), ldq, work, lanes, req_slot, req_start,   \
                           page_table, max_pages, static_cast<const bf16_t*>(kpool),               \
                           static_cast<const bf16_t*>(vpool), n_kv, qscale, part);                 \
        break;
    switch (G) {
        OUTLETS_DEC_G(1)
        OUTLETS_DEC_G(2)
        OUTLETS_DEC_G(4)
        OUTLETS_DEC_G(8)
    }
#undef OUTLETS_DEC_G
    hipLaunchKernelGGL(attn_decode_combine, dim3(n_req, (n_q + 7) / 8), dim3(256), 0, st, cu_segs, part, n_q,
                       static_cast<bf16_t*>(out), ldo, static_cast<const bf16_t*>(gate), ldq);
}

bool attn_supported(int n_q, int n_kv, int hd) {
    if (n_kv <= 0 || n_q % n_kv) return false;
    const int G = n_q / n_kv;
    return (G == 1 || G == 2 || G == 4 || G == 8) && (hd == 64 || hd == 128);
}

void launch_attn_paged(int act_fmt, int ntok, const void* q, int64_t ldq, void* out,
                       int64_t ldo, const int32_t* tok_slot, const int32_t* tok_pos,
                       const int32_t* page_table, int max_pages, const void* kpool,
                       const void* vpool, int n_q, int n_kv, int hd, const void* gate,
                       hipStream_t st) {
    if (ntok <= 0) return;
    const int G = n_q / n_kv;
    const float qscale = 1.4426950408889634f / sqrtf(static_cast<float>(hd));
    if (act_fmt == FMT_F32) {
        if (hd == 64) launch_hd<float, 64>(G, ntok, q, ldq, out, ldo, tok_slot, tok_pos, page_table, max_pages, kpool, vpool, n_kv, qscale, gate, st);
        else launch_hd<float, 128>(G, ntok, q, ldq, out, ldo, tok_slot, tok_pos, page_table, max_pages, kpool, vpool, n_kv, qscale, gate, st);
    } else {
        if (hd == 64) launch_hd<bf16_t, 64>(G, ntok, q, ldq, out, ldo, tok_slot, tok_pos, page_table, max_pages, kpool, vpool, n_kv, qscale, gate, st);
        else launch_hd<bf16_t, 128>(G, ntok, q, ldq, out, ldo, tok_slot, tok_pos, page_table, max_pages, kpool, vpool, n_kv, qscale, gate, st);
    }
}

}  // namespace outlets
