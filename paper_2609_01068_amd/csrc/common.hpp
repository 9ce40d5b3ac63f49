// Shared device helpers for the gfx950 kernels: storage formats, vector
// types for the MFMA builtins, and wave/block reductions (wavefront = 64).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace outlets {

typedef uint16_t bf16_t;  // bfloat16 storage (upper half of binary32)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// binary32 -> bfloat16, round to nearest even (inputs are finite).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<bf16_t>(u >> 16);
}

// Load/store one element in the activation storage format.
template <typename T> __device__ __forceinline__ float load_act(const T* p);
template <> __device__ __forceinline__ float load_act<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float load_act<bf16_t>(const bf16_t* p) { return bf16_to_f32(*p); }

template <typename T> __device__ __forceinline__ void store_act(T* p, float v);
template <> __device__ __forceinline__ void store_act<float>(float* p, float v) { *p = v; }
template <> __device__ __forceinline__ void store_act<bf16_t>(bf16_t* p, float v) { *p = f32_to_bf16(v); }

// Four OCP E4M3 codes (one dword) -> four bf16 (two packed dwords), using
// gfx950's hardware fp8 conversion (OCP encoding on this target).
__device__ __forceinline__ void e4m3x4_to_bf16x4(uint32_t codes, uint32_t& lo, uint32_t& hi) {
    // v_cvt_scalef32_pk_bf16_fp8 with scale 1: two OCP e4m3 codes (bytes 0-1,
    // or 2-3 with op_sel) to two bf16 in one instruction; every e4m3 value is
    // exactly representable in bf16, so the conversion is exact
    lo = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(codes, 1.0f, false));
    hi = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(codes, 1.0f, true));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

// Sum over a block of NT threads (NT a multiple of 64); every thread gets it.
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red) {
    v = wave_sum(v);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) red[w] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < NT / kWave; ++i) t += red[i];
    __syncthreads();
    return t;
}

}  // namespace outlets
