// Data movement of a bidirectional LSTM layer (section 4: the NMT encoder's
// first layer is bidirectional).  The reverse direction is an ordinary layer
// run on the time-reversed input, so its cache and gradients are in its own
// processing order s = T-1-t; these kernels convert at the layer's edges:
//   reverse  dst[s] = src[T-1-s] (any step size in 4-byte words)
//   join     out[t] = [h_fwd[t]; h_rev[T-1-t]]            ([T][2H][B])
//   split    dH_fwd[t] = dH[t][0:H], dH_rev[T-1-t] = dH[t][H:2H]
//   sum      dX[t] = dX_fwd[t] + dX_rev[T-1-t]
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace lstmss {

namespace {

__global__ __launch_bounds__(256) void reverse_kernel(const uint32_t *src, uint32_t *dst, int T,
                                                      long words) {
    const long n = (long)T * words, stride = (long)gridDim.x * 256;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += stride) {
        const long s = i / words, w = i - s * words;
        dst[i] = src[(T - 1 - s) * words + w];
    }
}

template <typename E>
__global__ __launch_bounds__(256) void join_kernel(const E *hf, const E *hr, E *out, int T,
                                                   long HB) {
    const long n = (long)T * 2 * HB, stride = (long)gridDim.x * 256;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += stride) {
        const long t = i / (2 * HB), e = i - t * 2 * HB;
        out[i] = e < HB ? hf[t * HB + e] : hr[(T - 1 - t) * HB + (e - HB)];
    }
}

__global__ __launch_bounds__(256) void split_kernel(const float *dH, float *df, float *dr, int T,
                                                    long HB) {
    const long n = (long)T * 2 * HB, stride = (long)gridDim.x * 256;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += stride) {
        const long t = i / (2 * HB), e = i - t * 2 * HB;
        if (e < HB)
            df[t * HB + e] = dH[i];
        else
            dr[(T - 1 - t) * HB + (e - HB)] = dH[i];
    }
}

__global__ __launch_bounds__(256) void sum_rev_kernel(const float *a, const float *b, float *out,
                                                      int T, long IB) {
    const long n = (long)T * IB, stride = (long)gridDim.x * 256;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += stride) {
        const long t = i / IB, e = i - t * IB;
        out[i] = a[i] + b[(T - 1 - t) * IB + e];
    }
}

unsigned grid_of(long n) { return (unsigned)std::max(1L, std::min(ceil_div(n, 256L), 8192L)); }

} // namespace

hipError_t launch_reverse(const void *src, void *dst, int T, long words, hipStream_t s) {
    if (T <= 0 || words <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(reverse_kernel, dim3(grid_of((long)T * words)), dim3(256), 0, s,
                       (const uint32_t *)src, (uint32_t *)dst, T, words);
    return hipGetLastError();
}

hipError_t launch_bidir_join(const void *hf, const void *hr, void *out, int T, long HB, bool bf16,
                             hipStream_t s) {
    const dim3 g(grid_of((long)T * 2 * HB));
    if (bf16)
        hipLaunchKernelGGL(join_kernel<uint16_t>, g, dim3(256), 0, s, (const uint16_t *)hf,
                           (const uint16_t *)hr, (uint16_t *)out, T, HB);
    else
        hipLaunchKernelGGL(join_kernel<uint32_t>, g, dim3(256), 0, s, (const uint32_t *)hf,
                           (const uint32_t *)hr, (uint32_t *)out, T, HB);
    return hipGetLastError();
}

hipError_t launch_bidir_split(const float *dH, float *df, float *dr, int T, long HB, hipStream_t s) {
    hipLaunchKernelGGL(split_kernel, dim3(grid_of((long)T * 2 * HB)), dim3(256), 0, s, dH, df, dr,
                       T, HB);
    return hipGetLastError();
}

hipError_t launch_sum_rev(const float *a, const float *b, float *out, int T, long IB,
                          hipStream_t s) {
    hipLaunchKernelGGL(sum_rev_kernel, dim3(grid_of((long)T * IB)), dim3(256), 0, s, a, b, out, T,
                       IB);
    return hipGetLastError();
}

} // namespace lstmss
