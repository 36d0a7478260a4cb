// Kernels of the training step around the sparsified backward pass: the
// loss gradient at the top of the stack and the SGD update of the weights.
//
// Paper: the models are trained by SGD with a fixed learning rate (section
// 4, experimental setup); dense-after-sparse training runs the first steps
// with the sparsified backward pass and the remaining steps dense (section
// 5, Table 2).  The loss is a synthetic regression loss on the top layer's
// hidden states (no dataset): L = (1 / 2B) sum (h - y)^2, dL/dh = (h - y) / B.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace lstmss {

namespace {

// W <- W - lr dW (formed in fp32, rounded to the storage type), b <- b - lr db.
template <typename TS>
__global__ __launch_bounds__(256) void sgd_kernel(TS *W, const float *dW, long nw, float *b,
                                                  const float *db, long nb, float lr) {
    const long stride = (long)gridDim.x * 256;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < nw; i += stride)
        st<TS>::store(W, i, st<TS>::load(W, i) - lr * dW[i]);
    if (b)
        for (long i = blockIdx.x * 256L + threadIdx.x; i < nb; i += stride)
            b[i] = b[i] - lr * db[i];
}

// dH = (h - y) / B; parts[block] = (1 / 2B) * (sum of this block's squared
// differences), each block summing its grid-stride elements in order and
// then its threads pairwise (fixed order: the result does not depend on
// timing).
template <typename TS>
__global__ __launch_bounds__(256) void mse_kernel(const TS *h, const float *y, float *dH, long n,
                                                  float inv_b, double *parts) {
    __shared__ double red[256];
    const long stride = (long)gridDim.x * 256;
    double acc = 0.0;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += stride) {
        const float df = st<TS>::load(h, i) - y[i];
        dH[i] = df * inv_b;
        acc += (double)df * (double)df;
    }
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if ((int)threadIdx.x < w)
            red[threadIdx.x] = red[threadIdx.x] + red[threadIdx.x + w];
        __syncthreads();
    }
    if (parts && threadIdx.x == 0)
        parts[blockIdx.x] = 0.5 * (double)inv_b * red[0];
}

// out = sum of parts[0, n) (n <= 1024), pairwise in a fixed order.
__global__ __launch_bounds__(1024) void sum_parts_kernel(const double *parts, int n, double *out) {
    __shared__ double red[1024];
    red[threadIdx.x] = (int)threadIdx.x < n ? parts[threadIdx.x] : 0.0;
    __syncthreads();
    for (int w = 512; w >= 1; w >>= 1) {
        if ((int)threadIdx.x < w)
            red[threadIdx.x] = red[threadIdx.x] + red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0)
        *out = red[0];
}

} // namespace

hipError_t launch_sgd(void *W, const float *dW, long nw, float *b, const float *db, long nb,
                      float lr, bool bf16, hipStream_t s) {
    const long n = std::max(nw, nb);
    if (n <= 0)
        return hipSuccess;
    const dim3 grid((unsigned)std::min(ceil_div(n, 256L), 8192L));
    if (bf16)
        hipLaunchKernelGGL(sgd_kernel<bf16_t>, grid, dim3(256), 0, s, (bf16_t *)W, dW, nw, b, db, nb, lr);
    else
        hipLaunchKernelGGL(sgd_kernel<float>, grid, dim3(256), 0, s, (float *)W, dW, nw, b, db, nb, lr);
    return hipGetLastError();
}

hipError_t launch_mse(const void *h, const float *y, float *dH, long n, float inv_b,
                      double *parts, int nparts, bool bf16, hipStream_t s) {
    if (n <= 0 || nparts < 1 || nparts > 1024)
        return hipErrorInvalidValue;
    if (bf16)
        hipLaunchKernelGGL(mse_kernel<bf16_t>, dim3(nparts), dim3(256), 0, s, (const bf16_t *)h, y, dH, n, inv_b, parts);
    else
        hipLaunchKernelGGL(mse_kernel<float>, dim3(nparts), dim3(256), 0, s, (const float *)h, y, dH, n, inv_b, parts);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !parts)
        return e;
    hipLaunchKernelGGL(sum_parts_kernel, dim3(1), dim3(1024), 0, s, parts, nparts, parts + nparts);
    return hipGetLastError();
}

} // namespace lstmss
