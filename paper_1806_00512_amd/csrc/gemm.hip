// The per-step weight-gradient product (for structures whose kept rows do
// not fit the time-batched kernel's routing tiles), the fused forward step
// of calls without a workspace, and the forward cell update.
//
// Paper: the weight gradient dW += dnet [x_t; h_{t-1}]^T of the kept slices
// (section 3, section 4); the forward computes the gate activations that
// the backward pass reads (section 4).
#include "gemm_common.h"

namespace lstmss {

namespace {

// --------------------------------------------------------------------------
// Weight gradient: dW[row(m)][n] += sum_b G[m][b] XH[n][b], XH = [x_t; h_{t-1}].
// Work-group tile 64 x 64 (4 waves, 2 x 2), batch staged 32 at a time.
// --------------------------------------------------------------------------
template <typename TS, bool SCATTER>
__global__ __launch_bounds__(THREADS) void gemm2_kernel(Gemm2Args a) {
    constexpr int TM = 64, TN = 64, TB = 32;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const long m0 = (long)blockIdx.x * TM;
    const int n0 = blockIdx.y * TN;
    const int B = a.B, I = a.I, NC = a.I + a.H;
    const TS *G = (const TS *)a.Gc;
    const TS *xt = (const TS *)a.xt;
    const TS *hp = (const TS *)a.hp;
    f32x16 acc;
    for (int v = 0; v < 16; ++v)
        acc[v] = 0.f;

    if constexpr (sizeof(TS) == 4) {
        __shared__ float As[TM][TB + 1];
        __shared__ float Bs[TN][TB + 1];
        for (int b0 = 0; b0 < B; b0 += TB) {
            for (int q = tid; q < TM * TB; q += THREADS) {
                const int mm = q / TB, bb = q % TB;
                const long m = m0 + mm;
                const int b = b0 + bb;
                As[mm][bb] = (m < a.Kp && b < B) ? G[m * B + b] : 0.f;
            }
            for (int q = tid; q < TN * TB; q += THREADS) {
                const int nn = q / TB, bb = q % TB;
                const int n = n0 + nn, b = b0 + bb;
                float v = 0.f;
                if (n < NC && b < B)
                    v = n < I ? xt[(long)n * B + b] : hp[(long)(n - I) * B + b];
                Bs[nn][bb] = v;
            }
            __syncthreads();
#pragma unroll
            for (int kk = 0; kk < TB; kk += 2) {
                const float av = As[wm * 32 + (lane & 31)][kk + (lane >> 5)];
                const float bv = Bs[wn * 32 + (lane & 31)][kk + (lane >> 5)];
                acc = mfma32x32x2(av, bv, acc);
            }
            __syncthreads();
        }
    } else {
        __shared__ __align__(16) uint16_t As[TM][TB + 8];
        __shared__ __align__(16) uint16_t Bs[TN][TB + 8];
        for (int b0 = 0; b0 < B; b0 += TB) {
            for (int q = tid; q < TM * TB; q += THREADS) {
                const int mm = q / TB, bb = q % TB;
                const long m = m0 + mm;
                const int b = b0 + bb;
                As[mm][bb] = (m < a.Kp && b < B) ? raw(G[m * B + b]) : (uint16_t)0;
            }
            for (int q = tid; q < TN * TB; q += THREADS) {
                const int nn = q / TB, bb = q % TB;
                const int n = n0 + nn, b = b0 + bb;
                uint16_t v = 0;
                if (n < NC && b < B)
                    v = raw(n < I ? xt[(long)n * B + b] : hp[(long)(n - I) * B + b]);
                Bs[nn][bb] = v;
            }
            __syncthreads();
#pragma unroll
            for (int kk = 0; kk < TB; kk += 16) {
                const u16x8 av = *(const u16x8 *)&As[wm * 32 + (lane & 31)][kk + 8 * (lane >> 5)];
                const u16x8 bv = *(const u16x8 *)&Bs[wn * 32 + (lane & 31)][kk + 8 * (lane >> 5)];
                acc = mfma32x32x16bf(av, bv, acc);
            }
            __syncthreads();
        }
    }

    const int n = n0 + wn * 32 + (lane & 31);
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const long m = m0 + wm * 32 + acc_row(lane, v);
        if (m < a.Kp && n < NC) {
            const long row = SCATTER ? (long)a.idx[m / a.P] * a.P + m % a.P : m;
            float *p = a.dW + row * NC + n;
            *p += acc[v];
        }
    }
}

// --------------------------------------------------------------------------
// Forward step.  Work-group: 32 hidden units x 32 batch columns; wave w
// computes gate w's pre-activations for those units, then the cell update
// runs from LDS.
// --------------------------------------------------------------------------
__device__ __forceinline__ float sigmoidf_(float x) { return 1.f / (1.f + __expf(-x)); }

template <typename TS>
__global__ __launch_bounds__(THREADS) void fwd_step_kernel(FwdArgs a) {
    constexpr int TK = 32;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int u0 = blockIdx.x * 32, n0 = blockIdx.y * 32;
    const int I = a.I, H = a.H, B = a.B, K = a.I + a.H;
    const TS *W = (const TS *)a.W;
    const TS *xt = (const TS *)a.xt;
    const TS *hp = (const TS *)a.hp;
    __shared__ float spre[4][32][33];
    f32x16 acc;
    for (int v = 0; v < 16; ++v)
        acc[v] = 0.f;

    if constexpr (sizeof(TS) == 4) {
        __shared__ float As[4 * 32][TK + 1];
        __shared__ float Bs[TK][32 + 4];
        for (int k0 = 0; k0 < K; k0 += TK) {
            for (int q = tid; q < 4 * 32 * TK; q += THREADS) {
                const int rr = q / TK, kk = q % TK;
                const int g = rr >> 5, u = u0 + (rr & 31), k = k0 + kk;
                As[rr][kk] = (u < H && k < K) ? W[((long)g * H + u) * K + k] : 0.f;
            }
            for (int q = tid; q < TK * 32; q += THREADS) {
                const int kk = q >> 5, nn = q & 31;
                const int k = k0 + kk, n = n0 + nn;
                float v = 0.f;
                if (k < K && n < B)
                    v = k < I ? xt[(long)k * B + n] : hp[(long)(k - I) * B + n];
                Bs[kk][nn] = v;
            }
            __syncthreads();
#pragma unroll
            for (int kk = 0; kk < TK; kk += 2) {
                const float av = As[wave * 32 + (lane & 31)][kk + (lane >> 5)];
                const float bv = Bs[kk + (lane >> 5)][lane & 31];
                acc = mfma32x32x2(av, bv, acc);
            }
            __syncthreads();
        }
    } else {
        __shared__ __align__(16) uint16_t As[4 * 32][TK + 8];
        __shared__ __align__(16) uint16_t Bs[32][TK + 8];
        for (int k0 = 0; k0 < K; k0 += TK) {
            for (int q = tid; q < 4 * 32 * TK; q += THREADS) {
                const int rr = q / TK, kk = q % TK;
                const int g = rr >> 5, u = u0 + (rr & 31), k = k0 + kk;
                As[rr][kk] = (u < H && k < K) ? raw(W[((long)g * H + u) * K + k]) : (uint16_t)0;
            }
            for (int q = tid; q < TK * 32; q += THREADS) {
                const int kk = q >> 5, nn = q & 31;
                const int k = k0 + kk, n = n0 + nn;
                uint16_t v = 0;
                if (k < K && n < B)
                    v = raw(k < I ? xt[(long)k * B + n] : hp[(long)(k - I) * B + n]);
                Bs[nn][kk] = v;
            }
            __syncthreads();
#pragma unroll
            for (int kk = 0; kk < TK; kk += 16) {
                const u16x8 av = *(const u16x8 *)&As[wave * 32 + (lane & 31)][kk + 8 * (lane >> 5)];
                const u16x8 bv = *(const u16x8 *)&Bs[lane & 31][kk + 8 * (lane >> 5)];
                acc = mfma32x32x16bf(av, bv, acc);
            }
            __syncthreads();
        }
    }

#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const int uu = acc_row(lane, v);
        const int u = u0 + uu;
        const float bias = (a.bias && u < H) ? a.bias[wave * H + u] : 0.f;
        spre[wave][uu][lane & 31] = acc[v] + bias;
    }
    __syncthreads();
    TS *gates = (TS *)a.gates;
    TS *hn = (TS *)a.hn;
    TS *hout = (TS *)a.hout;
    for (int q = tid; q < 32 * 32; q += THREADS) {
        const int uu = q >> 5, nn = q & 31;
        const int u = u0 + uu, n = n0 + nn;
        if (u >= H || n >= B)
            continue;
        const float ig = sigmoidf_(spre[0][uu][nn]);
        const float fg = sigmoidf_(spre[1][uu][nn]);
        const float gg = tanhf(spre[2][uu][nn]);
        const float og = sigmoidf_(spre[3][uu][nn]);
        const long e = (long)u * B + n;
        const float cv = fg * a.cp[e] + ig * gg;
        const float hv = og * tanhf(cv);
        a.cn[e] = cv;
        st<TS>::store(hn, e, hv);
        if (hout)
            st<TS>::store(hout, e, hv);
        st<TS>::store(gates, (long)(0 * H + u) * B + n, ig);
        st<TS>::store(gates, (long)(1 * H + u) * B + n, fg);
        st<TS>::store(gates, (long)(2 * H + u) * B + n, gg);
        st<TS>::store(gates, (long)(3 * H + u) * B + n, og);
    }
}

// Forward cell update of one step from the pre-activation pieces:
// a = zx + b + sum_s part[s] (input projection, bias, recurrent split-K
// partials); i, f, o = sigmoid, g = tanh; c = f c_prev + i g; h = o tanh(c).
// One thread per (unit, column); the stored gates and h are rounded to the
// storage type, c stays fp32 and is formed from the unrounded gates.
template <typename TS>
__global__ __launch_bounds__(256) void fwd_act_kernel(FwdActArgs a) {
    const long e = blockIdx.x * 256L + threadIdx.x;
    const long HB = (long)a.H * a.B;
    if (e >= HB)
        return;
    const int u = (int)(e / a.B), n = (int)(e - (long)u * a.B);
    float z[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const long r = (long)g * a.H + u;
        float v = a.zx[r * a.B + n] + (a.bias ? a.bias[r] : 0.f);
        for (int sp = 0; sp < a.nparts; ++sp)
            v += a.part[sp * a.part_stride + r * a.B + n];
        z[g] = v;
    }
    const float ig = sigmoidf_(z[0]), fg = sigmoidf_(z[1]), gg = tanhf(z[2]), og = sigmoidf_(z[3]);
    const float cv = fg * a.cp[e] + ig * gg;
    const float hv = og * tanhf(cv);
    a.cn[e] = cv;
    st<TS>::store((TS *)a.hn, e, hv);
    if (a.hout)
        st<TS>::store((TS *)a.hout, e, hv);
    TS *gates = (TS *)a.gates;
    st<TS>::store(gates, (long)(0 * a.H + u) * a.B + n, ig);
    st<TS>::store(gates, (long)(1 * a.H + u) * a.B + n, fg);
    st<TS>::store(gates, (long)(2 * a.H + u) * a.B + n, gg);
    st<TS>::store(gates, (long)(3 * a.H + u) * a.B + n, og);
}

} // namespace

hipError_t launch_fwd_act(const FwdActArgs &a, bool bf16, hipStream_t s) {
    const long HB = (long)a.H * a.B;
    if (HB <= 0)
        return hipSuccess;
    const dim3 grid((unsigned)ceil_div(HB, 256L));
    if (bf16)
        hipLaunchKernelGGL(fwd_act_kernel<bf16_t>, grid, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(fwd_act_kernel<float>, grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_gemm2(const Gemm2Args &a, bool bf16, hipStream_t s) {
    dim3 grid((unsigned)ceil_div(a.Kp, 64), (unsigned)ceil_div(a.I + a.H, 64));
    const bool scatter = a.idx != nullptr;
#define LSTMSS_G2(TS, SC) hipLaunchKernelGGL((gemm2_kernel<TS, SC>), grid, dim3(THREADS), 0, s, a)
    if (bf16) { if (scatter) LSTMSS_G2(bf16_t, true); else LSTMSS_G2(bf16_t, false); }
    else { if (scatter) LSTMSS_G2(float, true); else LSTMSS_G2(float, false); }
#undef LSTMSS_G2
    return hipGetLastError();
}

hipError_t launch_fwd_step(const FwdArgs &a, bool bf16, hipStream_t s) {
    dim3 grid((unsigned)ceil_div(a.H, 32), (unsigned)ceil_div(a.B, 32));
    if (bf16)
        hipLaunchKernelGGL(fwd_step_kernel<bf16_t>, grid, dim3(THREADS), 0, s, a);
    else
        hipLaunchKernelGGL(fwd_step_kernel<float>, grid, dim3(THREADS), 0, s, a);
    return hipGetLastError();
}

} // namespace lstmss
