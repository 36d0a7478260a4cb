// Pieces shared by the MFMA product kernels (data gradient, weight
// gradient, forward products): register staging vectors and the LDS / global
// address-space pointer types of the direct global -> LDS copies.
#pragma once

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace lstmss {

namespace {

constexpr int THREADS = 256;

__device__ __forceinline__ uint16_t raw(bf16_t v) { return v.bits; }

// Register staging of one global -> LDS vector: VW elements of a row.
template <typename TS, bool VEC>
struct Vec;
template <>
struct Vec<float, true> {
    static constexpr int W = 4;
    float v[4];
    __device__ __forceinline__ void load(const float *p, int valid) {
        if (valid >= 4) {
            const float4 t = *(const float4 *)p;
            v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                v[i] = i < valid ? p[i] : 0.f;
        }
    }
    __device__ __forceinline__ void zero() { v[0] = v[1] = v[2] = v[3] = 0.f; }
};
template <>
struct Vec<float, false> {
    static constexpr int W = 1;
    float v[1];
    __device__ __forceinline__ void load(const float *p, int valid) { v[0] = valid > 0 ? p[0] : 0.f; }
    __device__ __forceinline__ void zero() { v[0] = 0.f; }
};
template <>
struct Vec<bf16_t, true> {
    static constexpr int W = 8;
    uint16_t v[8];
    __device__ __forceinline__ void load(const bf16_t *p, int valid) {
        if (valid >= 8) {
            const u16x8 t = *(const u16x8 *)p;
#pragma unroll
            for (int i = 0; i < 8; ++i)
                v[i] = t[i];
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i)
                v[i] = i < valid ? p[i].bits : (uint16_t)0;
        }
    }
    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            v[i] = 0;
    }
};
template <>
struct Vec<bf16_t, false> {
    static constexpr int W = 1;
    uint16_t v[1];
    __device__ __forceinline__ void load(const bf16_t *p, int valid) { v[0] = valid > 0 ? p[0].bits : (uint16_t)0; }
    __device__ __forceinline__ void zero() { v[0] = 0; }
};

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glob_void_t;

} // namespace

} // namespace lstmss
