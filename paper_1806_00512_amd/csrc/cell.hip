// Backward elementwise gate-gradient kernel fused with structural
// sparsifying (score, per-region selection, compaction), plus the small
// helper kernels of the backward driver.
//
// Paper: section 3 (coarse-grained structural sparsifying of the gate
// gradient dnet, offset index array of the kept slices); the gate-gradient
// data flow is the one of Fig. 1 for the standard LSTM cell.
#include "common.h"
#include "kernels.h"

namespace lstmss {

namespace {

constexpr int CELL_THREADS = 256;

// Gate gradient of row r = g*H + u at batch column b for one backward step.
//   dh  = dH_up + dh_rec                       (dL/dh_t)
//   dc  = dc_t + dh * o * (1 - tanh(c_t)^2)    (dL/dc_t, unsparsified)
//   do  = dh * tanh(c_t) * o (1 - o)
//   di  = dc * g * i (1 - i)
//   df  = dc * c_{t-1} * f (1 - f)      and dc_{t-1} = dc * f
//   dg  = dc * i * (1 - g^2)
template <typename TS>
__device__ __forceinline__ float gate_grad(const CellArgs &a, const TS *gates, int g, int u, int b) {
    const int B = a.B, H = a.H;
    const int e = u * B + b;
    float dh = a.dH_up[e];
    for (int s = 0; s < a.dh_nparts; ++s)
        dh += a.dh_part[s * a.dh_stride + e];
    const float tc = tanhf(a.c_t[e]);
    const float o = st<TS>::load(gates, (3 * H + u) * B + b);
    if (g == 3)
        return dh * tc * o * (1.f - o);
    const float dcv = (a.dc_in ? a.dc_in[e] : 0.f) + dh * o * (1.f - tc * tc);
    if (g == 1) {
        const float f = st<TS>::load(gates, (H + u) * B + b);
        a.dc_out[e] = dcv * f;
        return dcv * a.c_prev[e] * f * (1.f - f);
    }
    const float i = st<TS>::load(gates, u * B + b);
    const float gg = st<TS>::load(gates, (2 * H + u) * B + b);
    if (g == 0)
        return dcv * gg * i * (1.f - i);
    return dcv * i * (1.f - gg * gg);
}

// True if slice i (score si) ranks above slice j (score sj) in a region.
__device__ __forceinline__ bool outranks(uint64_t ki, long i, uint64_t kj, long j) {
    return ki > kj || (ki == kj && i < j);
}

template <typename TS, int MODE>
__global__ __launch_bounds__(CELL_THREADS) void cell_select_kernel(CellArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int NW = CELL_THREADS / 64;
    const int B = a.B, P = a.P, R = a.R;
    const long G = 4L * a.H;

    // Reduction of the previous step's dX partial sums, spread over the grid.
    if (a.dx_out) {
        const long chunk = ceil_div(a.dx_n, gridDim.x);
        const long e0 = blockIdx.x * chunk, e1 = min(a.dx_n, e0 + chunk);
        for (long e = e0 + tid; e < e1; e += CELL_THREADS) {
            float s = 0.f;
            for (int p = 0; p < a.dx_nparts; ++p)
                s += a.dx_part[p * a.dx_stride + e];
            a.dx_out[e] = s;
        }
    }

    const long slices_per_wg = (long)a.regions_per_wg * R;
    const long j0 = blockIdx.x * slices_per_wg;
    if (j0 >= a.nslices)
        return;
    const int nsl = (int)min(slices_per_wg, a.nslices - j0);
    const long row0 = j0 * P;
    const int nrows = nsl * P;

    const TS *gates = (const TS *)a.gates;
    TS *dGc = (TS *)a.dGc;
    TS *dbg = (TS *)a.dbg;

    // LDS carve-up (sparse modes): dG rows, row sums of squares, row sums,
    // slice scores, keep flags, compacted slots.
    float *sdG = (float *)smem;
    double *srowsq = (double *)(smem + (((size_t)slices_per_wg * P * B * 4 + 15) & ~(size_t)15));
    float *srowsum = (float *)(srowsq + slices_per_wg * P);
    double *sscore = (double *)(((uintptr_t)(srowsum + slices_per_wg * P) + 15) & ~(uintptr_t)15);
    int *skeep = (int *)(sscore + slices_per_wg);
    int *sslot = skeep + slices_per_wg;

    // Phase 1: gate gradients, element-parallel over the work-group's rows
    // (all loads of an element are independent, so many are in flight).
    for (int q = tid; q < nrows * B; q += CELL_THREADS) {
        const int lr = q / B;
        const int b = q - lr * B;
        const int r = (int)row0 + lr;
        float v;
        if (MODE == CELL_GIVEN) {
            v = st<TS>::load((const TS *)a.dG_in, (long)r * B + b);
        } else {
            const int g = r / a.H;
            v = st<TS>::rnd(gate_grad<TS>(a, gates, g, r - g * a.H, b));
            if (dbg)
                st<TS>::store(dbg, r * B + b, v);
        }
        if (MODE == CELL_DENSE)
            st<TS>::store(dGc, r * B + b, v);
        sdG[q] = v;
    }
    __syncthreads();

    // Phase 1b: per-row sum of squares in the fixed order (partial l sums
    // b = l, l+64, ... in increasing b; partials combined by index xor 32, 16,
    // ..., 1).  With B <= 2^k < 64 every partial at index >= 2^k is zero and
    // adding it is exact, so 2^k lanes per row give the same value; a
    // wavefront then handles 64 / 2^k rows at once.  Row sums for the bias
    // gradient ride along.
    {
        int lpr = 1;
        while (lpr < B && lpr < 64)
            lpr <<= 1;
        const int rpw = 64 / lpr;
        const int sub = lane / lpr, sl = lane - sub * lpr;
        for (int base = wave * rpw; base < nrows; base += NW * rpw) {
            const int lr = base + sub;
            double part = 0.0;
            float rsum = 0.f;
            if (lr < nrows) {
                for (int b = sl; b < B; b += 64) {
                    const float v = sdG[lr * B + b];
                    part += (double)v * (double)v;
                    rsum += v;
                }
            }
            for (int off = lpr >> 1; off >= 1; off >>= 1) {
                if (MODE != CELL_DENSE)
                    part = part + shfl_xor_f64(part, off);
                rsum += shfl_xor_f32(rsum, off);
            }
            if (sl == 0 && lr < nrows) {
                if (MODE == CELL_DENSE) {
                    if (a.db)
                        a.db[row0 + lr] += rsum;
                } else {
                    srowsq[lr] = part;
                    srowsum[lr] = rsum;
                }
            }
        }
    }
    if (MODE == CELL_DENSE)
        return;
    __syncthreads();

    // Phase 2: slice scores, rows summed in increasing order.
    for (int j = tid; j < nsl; j += CELL_THREADS) {
        double s = srowsq[j * P];
        for (int p = 1; p < P; ++p)
            s = s + srowsq[j * P + p];
        sscore[j] = s;
        if (a.scores)
            a.scores[j0 + j] = s;
    }
    __syncthreads();

    // Phase 3: keep the R-S best slices of every region (a trailing region of
    // r < R slices keeps r - floor(S*r/R)); ties keep the lower index.
    for (int j = tid; j < nsl; j += CELL_THREADS) {
        const long gj = j0 + j;
        const long rs = (gj / R) * R;
        const long rlen = min((long)R, a.nslices - rs);
        const long nkeep = rlen - ((long)a.S * rlen) / R;
        const int ls = (int)(rs - j0);
        const uint64_t kj = score_key(sscore[j]);
        int beaten = 0;
        for (int i = ls; i < ls + rlen; ++i)
            if (i != j && outranks(score_key(sscore[i]), i, kj, j))
                ++beaten;
        skeep[j] = beaten < nkeep ? 1 : 0;
    }
    __syncthreads();

    // Phase 4: compacted slot = region * (R - S) + kept slices before it.
    for (int j = tid; j < nsl; j += CELL_THREADS) {
        const long gj = j0 + j;
        const long reg = gj / R;
        const int ls = (int)(reg * R - j0);
        int slot = -1;
        if (skeep[j]) {
            int pos = 0;
            for (int i = ls; i < j; ++i)
                pos += skeep[i];
            slot = (int)(reg * (R - a.S) + pos);
            a.idx[slot] = (int32_t)gj;
        }
        sslot[j] = slot;
    }
    __syncthreads();

    // Phase 5: copy kept rows to the compacted matrix; bias gradient.
    if (MODE == CELL_SPARSE || dGc) {
        for (long q = tid; q < (long)nrows * B; q += CELL_THREADS) {
            const int lr = (int)(q / B), b = (int)(q - (long)lr * B);
            const int slot = sslot[lr / P];
            if (slot >= 0)
                st<TS>::store(dGc, ((long)slot * P + lr % P) * B + b, sdG[q]);
        }
    }
    if (a.db) {
        for (int lr = tid; lr < nrows; lr += CELL_THREADS)
            if (sslot[lr / P] >= 0)
                a.db[row0 + lr] += srowsum[lr];
    }
    (void)G;
}

__global__ void fill_kernel(float *p, long n, float v) {
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void copy_in_kernel(float *dst, const float *src, long n) {
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
        dst[i] = src ? src[i] : 0.f;
}

__global__ void reduce_parts_kernel(float *out, const float *part, int nparts, long stride, long n) {
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) {
        float s = 0.f;
        for (int p = 0; p < nparts; ++p)
            s += part[p * stride + i];
        out[i] = s;
    }
}

template <typename TS>
__global__ void h0_store_kernel(TS *dst, const float *src, long n) {
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
        st<TS>::store(dst, i, src ? src[i] : 0.f);
}

int grid_for(long n) { return (int)max(1L, min(4096L, ceil_div(n, 256))); }

} // namespace

size_t cell_lds_bytes(const CellArgs &a, int mode) {
    (void)mode;
    const size_t spw = (size_t)a.regions_per_wg * a.R;
    const size_t rows = spw * a.P;
    size_t bytes = ((rows * a.B * 4 + 15) & ~(size_t)15);
    bytes += rows * 8 + rows * 4;
    bytes = (bytes + 15) & ~(size_t)15;
    bytes += spw * 8 + spw * 4 * 2;
    return bytes;
}

hipError_t launch_cell(const CellArgs &a, int mode, bool bf16, hipStream_t s) {
    const long spw = (long)a.regions_per_wg * a.R;
    const int grid = (int)ceil_div(a.nslices, spw);
    const size_t lds = cell_lds_bytes(a, mode);
#define LSTMSS_CELL(TS, M) \
    hipLaunchKernelGGL((cell_select_kernel<TS, M>), dim3(grid), dim3(CELL_THREADS), lds, s, a)
    if (bf16) {
        if (mode == CELL_DENSE) LSTMSS_CELL(bf16_t, CELL_DENSE);
        else if (mode == CELL_SPARSE) LSTMSS_CELL(bf16_t, CELL_SPARSE);
        else LSTMSS_CELL(bf16_t, CELL_GIVEN);
    } else {
        if (mode == CELL_DENSE) LSTMSS_CELL(float, CELL_DENSE);
        else if (mode == CELL_SPARSE) LSTMSS_CELL(float, CELL_SPARSE);
        else LSTMSS_CELL(float, CELL_GIVEN);
    }
#undef LSTMSS_CELL
    return hipGetLastError();
}

hipError_t launch_fill(float *p, long n, float v, hipStream_t s) {
    if (n <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(fill_kernel, dim3(grid_for(n)), dim3(256), 0, s, p, n, v);
    return hipGetLastError();
}

hipError_t launch_copy_in(float *dst, const float *src, long n, hipStream_t s) {
    if (n <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(copy_in_kernel, dim3(grid_for(n)), dim3(256), 0, s, dst, src, n);
    return hipGetLastError();
}

hipError_t launch_reduce_parts(float *out, const float *part, int nparts, long stride, long n,
                               hipStream_t s) {
    if (n <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(reduce_parts_kernel, dim3(grid_for(n)), dim3(256), 0, s, out, part, nparts,
                       stride, n);
    return hipGetLastError();
}

hipError_t launch_h0_store(void *dst, const float *src, long n, bool bf16, hipStream_t s) {
    if (n <= 0)
        return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL(h0_store_kernel<bf16_t>, dim3(grid_for(n)), dim3(256), 0, s,
                           (bf16_t *)dst, src, n);
    else
        hipLaunchKernelGGL(h0_store_kernel<float>, dim3(grid_for(n)), dim3(256), 0, s,
                           (float *)dst, src, n);
    return hipGetLastError();
}

} // namespace lstmss
