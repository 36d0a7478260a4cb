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

// Work-group barrier for LDS traffic: this wavefront's LDS operations are
// complete, then all wavefronts meet.  Unlike __syncthreads() it does not
// wait for outstanding global loads (whose release fence would drain a
// multi-stage global -> LDS copy pipeline); the callers wait for the copies a
// stage needs with explicit vmcnt waits before it.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// One global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4): lane
// j writes bytes [16 j, 16 j + 16) of the 1 KB LDS block at lds_dst (the
// same block for the whole wavefront).  Issued as inline assembly so that the
// compiler does not take it for an LDS store that every later LDS read has
// to wait for (it would drain the copy pipeline before each stage's reads);
// callers order it with explicit vmcnt waits and lds_barrier().  It sets m0,
// which the kernels using it hold nothing else in (no other m0 use in their
// code).
__device__ __forceinline__ void dma16(const void *gsrc, lds_void_t *lds_dst) {
    const int lds = __builtin_amdgcn_readfirstlane((int)(uintptr_t)lds_dst);
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(gsrc), "s"(lds)
                 : "memory", "m0");
}

// The same for 4 bytes per lane (global_load_lds_dword): lane j writes bytes
// [4 j, 4 j + 4) of the 256-byte LDS block at lds_dst.
__device__ __forceinline__ void dma4(const void *gsrc, lds_void_t *lds_dst) {
    const int lds = __builtin_amdgcn_readfirstlane((int)(uintptr_t)lds_dst);
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off"
                 :
                 : "v"(gsrc), "s"(lds)
                 : "memory", "m0");
}

// s_waitcnt immediate that waits until at most n vector-memory operations of
// this wavefront are outstanding (the other counters left at their maxima).
// Buffer resource of raw bytes from base (gfx9 layout: stride 0,
// `bytes` records, the data-format word of untyped buffer access).
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4 buf_rsrc(const void *base, uint32_t bytes) {
    const uint64_t p = (uint64_t)(uintptr_t)base;
    i32x4 r;
    r[0] = (int)(uint32_t)p;
    r[1] = (int)((uint32_t)(p >> 32) & 0xffffu);
    r[2] = (int)bytes;
    r[3] = 0x00020000;
    return r;
}

// dma16 through a buffer resource: lane j copies the 16 bytes at
// base + soff + voff (voff its own byte offset) to bytes [16 j, 16 j + 16) of
// the 1 KB LDS block at lds_dst.  Only the 32-bit offset lives in a vector
// register.  Same ordering rules as dma16.
__device__ __forceinline__ void dma16_buf(i32x4 rsrc, int voff, int soff, lds_void_t *lds_dst) {
    const int lds = __builtin_amdgcn_readfirstlane((int)(uintptr_t)lds_dst);
    asm volatile("s_mov_b32 m0, %1\n\tbuffer_load_dwordx4 %0, %2, %3 offen lds"
                 :
                 : "v"(voff), "s"(lds), "s"(rsrc), "s"(soff)
                 : "memory", "m0");
}

constexpr int vmcnt_imm(int n) { return (n & 0xf) | ((n >> 4) << 14) | (0x7 << 4) | (0xf << 8); }

} // namespace

} // namespace lstmss
