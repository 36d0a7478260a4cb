// Internal device helpers shared by the lstmss kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lstmss {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

// bf16 is kept as raw 16-bit patterns in memory.
struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round to nearest bf16, ties to even; NaN stays NaN (quiet).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Storage-type traits: load as float, store from float, and the value a
// float takes once stored (identity for fp32, rounding for bf16).
template <typename TS>
struct st;

template <>
struct st<float> {
    static constexpr int bytes = 4;
    __device__ __forceinline__ static float load(const float *p, long i) { return p[i]; }
    __device__ __forceinline__ static void store(float *p, long i, float v) { p[i] = v; }
    __device__ __forceinline__ static float rnd(float v) { return v; }
};

template <>
struct st<bf16_t> {
    static constexpr int bytes = 2;
    __device__ __forceinline__ static float load(const bf16_t *p, long i) { return bf16_to_f32(p[i].bits); }
    __device__ __forceinline__ static void store(bf16_t *p, long i, float v) { p[i].bits = f32_to_bf16(v); }
    __device__ __forceinline__ static float rnd(float v) { return bf16_to_f32(f32_to_bf16(v)); }
};

__device__ __forceinline__ f32x16 mfma32x32x2(float a, float b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 mfma32x32x16bf(u16x8 a, u16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Accumulator layout of a 32x32 MFMA tile: lane l, register v holds
// row 8*(v/4) + 4*(l/32) + (v%4), column l%32.
__device__ __forceinline__ int acc_row(int lane, int v) { return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3); }

__device__ __forceinline__ double shfl_xor_f64(double v, int mask) { return __shfl_xor(v, mask, 64); }
__device__ __forceinline__ float shfl_xor_f32(float v, int mask) { return __shfl_xor(v, mask, 64); }

// Total-order key for non-negative scores: NaN above +inf above finite.
__device__ __forceinline__ uint64_t score_key(double s) {
    if (s != s)
        return ~0ull;
    return (uint64_t)__double_as_longlong(s);
}

__host__ __device__ __forceinline__ long ceil_div(long a, long b) { return (a + b - 1) / b; }

// init + p[0] + p[stride] + ... + p[(n-1)*stride], added in that order; the
// loads are issued NB at a time so their latencies overlap.
template <int NB = 8>
__device__ __forceinline__ float sum_parts(float init, const float *p, int n, long stride) {
    float s = init;
    int i = 0;
    for (; i + NB <= n; i += NB) {
        float v[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j)
            v[j] = p[(long)(i + j) * stride];
#pragma unroll
        for (int j = 0; j < NB; ++j)
            s += v[j];
    }
    if (i < n) {
        float v[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j)
            v[j] = i + j < n ? p[(long)(i + j) * stride] : 0.f;
#pragma unroll
        for (int j = 0; j < NB; ++j)
            if (i + j < n)
                s += v[j];
    }
    return s;
}

} // namespace lstmss
