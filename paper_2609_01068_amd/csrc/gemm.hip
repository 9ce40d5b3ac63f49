// Dense contractions of the draft layer and the length head on gfx950.
//
// bf16 / e4m3-weight path: 256x256x64 workgroup tiles, 4 waves (2 x 2), each
// wave owning a 128x128 sub-tile built from v_mfma_f32_32x32x16_bf16 (its 256
// accumulators fit the accumulation registers at one wave per SIMD).  Tiles
// are staged through LDS, double buffered with a register prefetch of the
// next K slice, so each iteration needs a single barrier.  LDS rows are 64
// bf16 (128 B) with 16-byte chunks XOR-swizzled by (row / 2) % 8, which makes
// the 16-lane phases of ds_read_b128 fragment loads conflict free.  e4m3
// weights are widened to bf16 (exact) on their way into LDS and the per-row
// scale is applied in the epilogue.
//
// fp32 path (tiny shape): a plain LDS-tiled VALU kernel with full bounds
// handling; it exists for the fp32 configuration, not for speed.
#include "common.hpp"
#include "kernels.hpp"
#include "outlets.h"

namespace outlets {

namespace {

constexpr int BK = 64;

__device__ __forceinline__ int swz(int row, int c) { return row * 8 + (c ^ ((row >> 1) & 7)); }

// logical B row -> (block, physical row)
__device__ __forceinline__ void b_row(const GemmB& B, int n, int& s, int& r) {
    if (B.paired) {
        int blk = n >> 5;
        s = blk & 1;
        r = (blk >> 1) * 32 + (n & 31);
    } else {
        s = (n >= B.nend[0]) + (n >= B.nend[1]);
        r = n - (s == 0 ? 0 : B.nend[s - 1]);
    }
}

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

// Map the hardware workgroup id to a tile so that consecutive tiles run on
// the same XCD (workgroups are dealt round-robin over the 8 XCDs) and walk
// GM row-tiles before moving along N, so A rows and B columns are reused
// from that XCD's L2.
__device__ __forceinline__ void tile_of(int bid, int nb, int mt, int nt, int& tm, int& tn) {
    const int q = nb / 8, r = nb % 8;
    const int x = bid % 8, i = bid / 8;
    const int pid = (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
    constexpr int GM = 8;
    const int group = pid / (GM * nt);
    const int first = group * GM;
    const int gsize = min(mt - first, GM);
    const int in = pid % (GM * nt);
    tm = first + in % gsize;
    tn = in / gsize;
}

template <int EPI, bool E4M3, typename OutT>
__global__ void __launch_bounds__(256)
gemm_mfma_256x256(int M, int N, int K, GemmA A, GemmB B, GemmC C, int k_per_split) {
    constexpr int BM = 256, BN = 256, NT = 256;
    constexpr int WN = 2;
    constexpr int TM = 128, TN = 128, FM = TM / 32, FN = TN / 32;
    constexpr int RPP = NT / 8;             // tile rows covered per load pass
    constexpr int CA = BM / RPP;            // 16-byte A chunks per thread
    constexpr int CB = BN / RPP;
    __shared__ uint4 lds[2][(BM + BN) * (BK / 8)];

    const int mt = (M + BM - 1) / BM, nt = N / BN;
    int tm, tn;
    tile_of(blockIdx.x, mt * nt, mt, nt, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int kb = blockIdx.y * k_per_split;
    const int ke = min(K, kb + k_per_split);
    const int nk = (ke - kb) / BK;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int chunk = tid & 7, r0 = tid >> 3;

    // A: thread rows r0 + RPP * i, clamped to the last valid row
    const bf16_t* a_base = static_cast<const bf16_t*>(A.p[0]) + (int64_t)min(m0 + r0, M - 1) * A.ld + chunk * 8;
    const int a_room = M - 1 - (m0 + r0);   // rows available below r0 (may be < 0 on the last tile)
    const int64_t seg1 = (const bf16_t*)A.p[1] - (const bf16_t*)A.p[0];
    const int64_t seg2 = (const bf16_t*)A.p[2] - (const bf16_t*)A.p[0];
    // B: thread rows r0 + RPP * i.  Rows of one 256-row tile stay in one block
    // (block ends are multiples of 256); in paired mode consecutive 32-row
    // passes alternate gate/up, so chunk i reads bsrc[i & 1] + (i >> 1) * bstep.
    const char* bsrc[2];
    int64_t bstep;
    {
        const int esz = E4M3 ? 1 : 2;
        int s, r;
        b_row(B, n0 + r0, s, r);
        bsrc[0] = static_cast<const char*>(B.p[s]) + ((int64_t)r * B.ld + chunk * 8) * esz;
        if (B.paired) {
            int s1, r1;
            b_row(B, n0 + r0 + RPP, s1, r1);
            bsrc[1] = static_cast<const char*>(B.p[s1]) + ((int64_t)r1 * B.ld + chunk * 8) * esz;
            bstep = (int64_t)RPP * B.ld * esz;
        } else {
            bsrc[1] = bsrc[0] + (int64_t)RPP * B.ld * esz;
            bstep = (int64_t)2 * RPP * B.ld * esz;
        }
    }

    uint4 ra[CA], rb[CB];
    auto gload = [&](int k0) {
        const int s = k0 / A.kseg;
        const int64_t aoff = (s == 0 ? 0 : (s == 1 ? seg1 : seg2)) + (k0 - s * A.kseg);
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const int dr = max(0, min(RPP * i, a_room));
            ra[i] = *reinterpret_cast<const uint4*>(a_base + aoff + (int64_t)dr * A.ld);
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const char* src = bsrc[i & 1] + (i >> 1) * bstep;
            if (E4M3) {
                uint2 c8 = *reinterpret_cast<const uint2*>(src + k0);
                uint32_t x0, x1, x2, x3;
                e4m3x4_to_bf16x4(c8.x, x0, x1);
                e4m3x4_to_bf16x4(c8.y, x2, x3);
                rb[i] = make_uint4(x0, x1, x2, x3);
            } else {
                rb[i] = *reinterpret_cast<const uint4*>(src + (int64_t)k0 * 2);
            }
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < CA; ++i) lds[buf][swz(r0 + RPP * i, chunk)] = ra[i];
#pragma unroll
        for (int i = 0; i < CB; ++i) lds[buf][BM * 8 + swz(r0 + RPP * i, chunk)] = rb[i];
    };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    if (nk > 0) {
        gload(kb);
        lstore(0);
    }
    __syncthreads();
    const int half = lane >> 5, l32 = lane & 31;
    for (int it = 0; it < nk; ++it) {
        const int buf = it & 1;
        if (it + 1 < nk) gload(kb + (it + 1) * BK);
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            const int c = kk * 2 + half;
            bf16x8 af[FM], bfr[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                int row = wm * TM + i * 32 + l32;
                uint4 v = lds[buf][swz(row, c)];
                af[i] = __builtin_bit_cast(bf16x8, v);
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                int row = wn * TN + j * 32 + l32;
                uint4 v = lds[buf][BM * 8 + swz(row, c)];
                bfr[j] = __builtin_bit_cast(bf16x8, v);
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
        if (it + 1 < nk) lstore(buf ^ 1);
        __syncthreads();
    }

    // epilogue: lane holds column l32 of each 32x32 block, rows
    // 8*(r/4) + 4*half + r%4 for accumulator element r
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int n = n0 + wn * TN + j * 32 + l32;
        float sc = 1.f;
        if (E4M3) {
            int s, r;
            b_row(B, n, s, r);
            sc = bf16_to_f32(B.scale[s][r]);
        }
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = m0 + wm * TM + i * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
                if (m >= M) continue;
                float v = acc[i][j][r] * sc;
                if (EPI == EPI_STORE_F32) {
                    static_cast<float*>(C.c)[(int64_t)m * C.ldc + n] = v;
                } else if (EPI == EPI_STORE_ACT) {
                    store_act<OutT>(static_cast<OutT*>(C.c) + (int64_t)m * C.ldc + n, v);
                } else if (EPI == EPI_RESID_F32) {
                    static_cast<float*>(C.c)[(int64_t)m * C.ldc + n] = C.resid[(int64_t)m * C.ldr + n] + v;
                } else if (EPI == EPI_PARTIAL) {
                    static_cast<float*>(C.c)[blockIdx.y * C.split_stride + (int64_t)m * C.ldc + n] = v;
                } else if (EPI == EPI_SWIGLU) {
                    if ((j & 1) == 0) {
                        // partner fragment j + 1 holds the matching up column
                        float sc_u = 1.f;
                        if (E4M3) {
                            int s, rr;
                            b_row(B, n + 32, s, rr);
                            sc_u = bf16_to_f32(B.scale[s][rr]);
                        }
                        const float g = v, u = acc[i][j + 1][r] * sc_u;
                        const int f = ((n >> 5) >> 1) * 32 + l32;
                        store_act<OutT>(static_cast<OutT*>(C.c) + (int64_t)m * C.ldc + f, silu_f(g) * u);
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------- fp32 VALU path
template <int EPI>
__global__ void __launch_bounds__(256)
gemm_f32_64x64(int M, int N, int K, GemmA A, GemmB B, GemmC C, int k_per_split) {
    // EPI_SWIGLU: logical N is the number of features; each output needs the
    // gate row (p[0]) and the up row (p[1]).
    constexpr int T = 64, KT = 16;
    constexpr bool DUAL = (EPI == EPI_SWIGLU);
    __shared__ float sa[KT][T + 1];
    __shared__ float sb[DUAL ? 2 : 1][KT][T + 1];
    const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
    const int m0 = blockIdx.x * T, n0 = blockIdx.z * T;
    const int kb = blockIdx.y * k_per_split, ke = min(K, kb + k_per_split);
    float acc[DUAL ? 2 : 1][4][4] = {};
    for (int k0 = kb; k0 < ke; k0 += KT) {
        for (int e = threadIdx.x; e < T * KT; e += 256) {
            int r = e / KT, kk = e % KT, m = m0 + r, k = k0 + kk;
            float v = 0.f;
            if (m < M && k < ke) {
                int s = k / A.kseg;
                v = static_cast<const float*>(A.p[s])[(int64_t)m * A.ld + (k - s * A.kseg)];
            }
            sa[kk][r] = v;
            int n = n0 + r;
#pragma unroll
            for (int q = 0; q < (DUAL ? 2 : 1); ++q) {
                float w = 0.f;
                if (n < N && k < ke) {
                    int s, rr;
                    if (DUAL) { s = q; rr = n; } else { b_row(B, n, s, rr); }
                    w = static_cast<const float*>(B.p[s])[(int64_t)rr * B.ld + k];
                }
                sb[q][kk][r] = w;
            }
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < KT; ++kk) {
            float av[4], bv[DUAL ? 2 : 1][4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = sa[kk][ty * 4 + i];
#pragma unroll
            for (int q = 0; q < (DUAL ? 2 : 1); ++q)
#pragma unroll
                for (int j = 0; j < 4; ++j) bv[q][j] = sb[q][kk][tx * 4 + j];
#pragma unroll
            for (int q = 0; q < (DUAL ? 2 : 1); ++q)
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[q][i][j] = fmaf(av[i], bv[q][j], acc[q][i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        int m = m0 + ty * 4 + i;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            int n = n0 + tx * 4 + j;
            if (n >= N) continue;
            float v = acc[0][i][j];
            float* c = static_cast<float*>(C.c);
            if (EPI == EPI_STORE_F32 || EPI == EPI_STORE_ACT) c[(int64_t)m * C.ldc + n] = v;
            else if (EPI == EPI_RESID_F32) c[(int64_t)m * C.ldc + n] = C.resid[(int64_t)m * C.ldr + n] + v;
            else if (EPI == EPI_PARTIAL) c[blockIdx.y * C.split_stride + (int64_t)m * C.ldc + n] = v;
            else if (EPI == EPI_SWIGLU) {
                float g = v, u = acc[DUAL ? 1 : 0][i][j];
                c[(int64_t)m * C.ldc + n] = g / (1.0f + expf(-g)) * u;
            }
        }
    }
}

template <int EPI, bool E4M3>
void launch_mfma(int act_fmt, int M, int N, int K, const GemmA& a, const GemmB& b,
                 const GemmC& c, int splits, hipStream_t st) {
    (void)act_fmt;
    const int mt = (M + 255) / 256, nt = N / 256;
    const int kps = ((K / BK + splits - 1) / splits) * BK;
    dim3 grid(mt * nt, splits);
    hipLaunchKernelGGL((gemm_mfma_256x256<EPI, E4M3, bf16_t>), grid, dim3(256), 0, st, M, N, K,
                       a, b, c, kps);
}

template <int EPI>
void launch_f32(int M, int N, int K, const GemmA& a, const GemmB& b, const GemmC& c, int splits,
                hipStream_t st) {
    const int kps = ((K + splits - 1) / splits + 15) / 16 * 16;
    dim3 grid((M + 63) / 64, splits, (N + 63) / 64);
    hipLaunchKernelGGL((gemm_f32_64x64<EPI>), grid, dim3(256), 0, st, M, N, K, a, b, c, kps);
}

}  // namespace

int gemm_check(int act_fmt, int w_fmt, int epi, int M, int N, int K, const GemmA& a,
               const GemmB& b, int splits, const char** why) {
    if (M <= 0 || N <= 0 || K <= 0 || splits <= 0) { *why = "gemm: empty shape"; return OUTLETS_ERR_INVALID_ARG; }
    if (w_fmt == FMT_F32) {
        if (act_fmt != FMT_F32) { *why = "gemm: f32 weights need f32 activations"; return OUTLETS_ERR_UNSUPPORTED; }
        if (epi == EPI_SWIGLU && b.paired) { *why = "gemm: f32 swiglu uses dual rows"; return OUTLETS_ERR_UNSUPPORTED; }
        return OUTLETS_OK;
    }
    if (act_fmt != FMT_BF16) { *why = "gemm: bf16/e4m3 weights need bf16 activations"; return OUTLETS_ERR_UNSUPPORTED; }
    if (N % 256) { *why = "gemm: N must be a multiple of 256"; return OUTLETS_ERR_UNSUPPORTED; }
    if (K % BK || a.kseg % BK) { *why = "gemm: K must be a multiple of 64"; return OUTLETS_ERR_UNSUPPORTED; }
    if ((K / BK) < splits) { *why = "gemm: more K splits than K tiles"; return OUTLETS_ERR_UNSUPPORTED; }
    if (a.ld % 8 || b.ld % (w_fmt == FMT_E4M3 ? 16 : 8)) { *why = "gemm: row strides must keep 16-byte alignment"; return OUTLETS_ERR_UNSUPPORTED; }
    for (int s = 0; s < 3; ++s) {
        if (a.p[s] && (reinterpret_cast<uintptr_t>(a.p[s]) & 15)) { *why = "gemm: A must be 16-byte aligned"; return OUTLETS_ERR_UNSUPPORTED; }
        if (b.p[s] && (reinterpret_cast<uintptr_t>(b.p[s]) & 15)) { *why = "gemm: B must be 16-byte aligned"; return OUTLETS_ERR_UNSUPPORTED; }
    }
    if (!b.paired)
        for (int s = 0; s < 2; ++s)
            if (b.nend[s] % 256) { *why = "gemm: B row blocks must be multiples of 256"; return OUTLETS_ERR_UNSUPPORTED; }
    if (epi == EPI_SWIGLU && !b.paired) { *why = "gemm: swiglu needs paired gate/up rows"; return OUTLETS_ERR_UNSUPPORTED; }
    return OUTLETS_OK;
}

void gemm_launch(int act_fmt, int w_fmt, int epi, int M, int N, int K, const GemmA& a,
                 const GemmB& b, const GemmC& c, int splits, hipStream_t st) {
    if (w_fmt == FMT_F32) {
        switch (epi) {
            case EPI_STORE_F32: case EPI_STORE_ACT: launch_f32<EPI_STORE_F32>(M, N, K, a, b, c, splits, st); break;
            case EPI_RESID_F32: launch_f32<EPI_RESID_F32>(M, N, K, a, b, c, splits, st); break;
            case EPI_SWIGLU: launch_f32<EPI_SWIGLU>(M, N, K, a, b, c, splits, st); break;
            case EPI_PARTIAL: launch_f32<EPI_PARTIAL>(M, N, K, a, b, c, splits, st); break;
        }
        return;
    }
    const bool e4 = (w_fmt == FMT_E4M3);
#define OUTLETS_GEMM_CASE(E)                                                        \
    case E:                                                                         \
        if (e4) launch_mfma<E, true>(act_fmt, M, N, K, a, b, c, splits, st);        \
        else launch_mfma<E, false>(act_fmt, M, N, K, a, b, c, splits, st);          \
        break;
    switch (epi) {
        OUTLETS_GEMM_CASE(EPI_STORE_F32)
        OUTLETS_GEMM_CASE(EPI_STORE_ACT)
        OUTLETS_GEMM_CASE(EPI_RESID_F32)
        OUTLETS_GEMM_CASE(EPI_SWIGLU)
        OUTLETS_GEMM_CASE(EPI_PARTIAL)
    }
#undef OUTLETS_GEMM_CASE
}

}  // namespace outlets
