// MFMA GEMMs of the backward pass on the compacted gate gradient, and the
// fused forward step.
//
// Paper: the gate gradient feeds every weight and data gradient product of
// the LSTM backward pass (section 3); after sparsifying, the kept slices are
// a dense matrix plus an offset index array, so the products run as dense
// block GEMMs that read the kept rows of W through the index (section 3 after
// Fig. 2, section 4).  Here:
//   data gradient    [dx_t; dh_{t-1}] = W_c^T dG_c   (W_c = kept rows of W)
//   weight gradient  dW[kept rows]   += dG_c [x_t; h_{t-1}]^T
//
// Tiles are 64-wide-wavefront MFMA tiles (32x32 outputs per wave), staged
// through LDS.  fp32 uses v_mfma_f32_32x32x2f32; bf16 uses
// v_mfma_f32_32x32x16_bf16 with fp32 accumulation.
#include "common.h"
#include "kernels.h"

namespace lstmss {

namespace {

constexpr int THREADS = 256;

__device__ __forceinline__ uint16_t raw(bf16_t v) { return v.bits; }

// --------------------------------------------------------------------------
// Data gradient: part[z][m][n] = sum over k in split z of W[row(k)][m] G[k][n]
// where row(k) = idx[k/P]*P + k%P (kept rows) or k (dense).
// Work-group tile TM x TN (4 waves, 32x32 each), K staged TK at a time.
// --------------------------------------------------------------------------
template <typename TS, int TN, bool GATHER>
__global__ __launch_bounds__(THREADS) void gemm1_kernel(Gemm1Args a) {
    constexpr int TM = 4096 / TN;
    constexpr int TK = GEMM1_TK;
    constexpr int WM = TM / 32;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int mm0 = blockIdx.x * TM;
    const int n0 = blockIdx.y * TN;
    const long kb = blockIdx.z * a.k_chunk;
    const long ke = min(a.Kp, kb + a.k_chunk);
    const int M = a.M, N = a.N;
    const TS *W = (const TS *)a.W;
    const TS *G = (const TS *)a.Gc;
    f32x16 acc;
    for (int v = 0; v < 16; ++v)
        acc[v] = 0.f;

    if constexpr (sizeof(TS) == 4) {
        // fp32: LDS as [k][row]; lanes 0-31 read k, lanes 32-63 read k+1.
        __shared__ float As[TK][TM + 4];
        __shared__ float Bs[TK][TN + 4];
        for (long k0 = kb; k0 < ke; k0 += TK) {
            for (int q = tid; q < TK * TM; q += THREADS) {
                const int kk = q / TM, mm = q % TM;
                const long k = k0 + kk;
                const int m = a.m_begin + mm0 + mm;
                float v = 0.f;
                if (k < ke && m < M) {
                    const long row = GATHER ? (long)a.idx[k / a.P] * a.P + k % a.P : k;
                    v = W[row * a.ldw + m];
                }
                As[kk][mm] = v;
            }
            for (int q = tid; q < TK * TN; q += THREADS) {
                const int kk = q / TN, nn = q % TN;
                const long k = k0 + kk;
                const int n = n0 + nn;
                Bs[kk][nn] = (k < ke && n < N) ? G[k * N + n] : 0.f;
            }
            __syncthreads();
#pragma unroll
            for (int kk = 0; kk < TK; kk += 2) {
                const float av = As[kk + (lane >> 5)][wm * 32 + (lane & 31)];
                const float bv = Bs[kk + (lane >> 5)][wn * 32 + (lane & 31)];
                acc = mfma32x32x2(av, bv, acc);
            }
            __syncthreads();
        }
    } else {
        // bf16: LDS as [row][k] so each lane reads 8 consecutive k (16 bytes).
        __shared__ __align__(16) uint16_t As[TM][TK + 8];
        __shared__ __align__(16) uint16_t Bs[TN][TK + 8];
        for (long k0 = kb; k0 < ke; k0 += TK) {
            for (int q = tid; q < TK * TM; q += THREADS) {
                const int kk = q / TM, mm = q % TM;
                const long k = k0 + kk;
                const int m = a.m_begin + mm0 + mm;
                uint16_t v = 0;
                if (k < ke && m < M) {
                    const long row = GATHER ? (long)a.idx[k / a.P] * a.P + k % a.P : k;
                    v = raw(W[row * a.ldw + m]);
                }
                As[mm][kk] = v;
            }
            for (int q = tid; q < TK * TN; q += THREADS) {
                const int kk = q / TN, nn = q % TN;
                const long k = k0 + kk;
                const int n = n0 + nn;
                Bs[nn][kk] = (k < ke && n < N) ? raw(G[k * N + n]) : (uint16_t)0;
            }
            __syncthreads();
#pragma unroll
            for (int kk = 0; kk < TK; kk += 16) {
                const u16x8 av = *(const u16x8 *)&As[wm * 32 + (lane & 31)][kk + 8 * (lane >> 5)];
                const u16x8 bv = *(const u16x8 *)&Bs[wn * 32 + (lane & 31)][kk + 8 * (lane >> 5)];
                acc = mfma32x32x16bf(av, bv, acc);
            }
            __syncthreads();
        }
    }

    float *out = a.part + blockIdx.z * a.part_stride;
    const int n = n0 + wn * 32 + (lane & 31);
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const int m = a.m_begin + mm0 + wm * 32 + acc_row(lane, v);
        if (m < M && n < N)
            out[(long)m * N + n] = acc[v];
    }
}

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

} // namespace

int gemm1_tn(int N) { return N <= 32 ? 32 : 64; }
int gemm1_tm(int N) { return 4096 / gemm1_tn(N); }

hipError_t launch_gemm1(const Gemm1Args &a, bool bf16, hipStream_t s) {
    const int TN = gemm1_tn(a.N), TM = 4096 / TN;
    dim3 grid((unsigned)ceil_div(a.M - a.m_begin, TM), (unsigned)ceil_div(a.N, TN), (unsigned)a.splitk);
    const bool gather = a.idx != nullptr;
#define LSTMSS_G1(TS, TNV, GA) hipLaunchKernelGGL((gemm1_kernel<TS, TNV, GA>), grid, dim3(THREADS), 0, s, a)
    if (bf16) {
        if (TN == 32) { if (gather) LSTMSS_G1(bf16_t, 32, true); else LSTMSS_G1(bf16_t, 32, false); }
        else { if (gather) LSTMSS_G1(bf16_t, 64, true); else LSTMSS_G1(bf16_t, 64, false); }
    } else {
        if (TN == 32) { if (gather) LSTMSS_G1(float, 32, true); else LSTMSS_G1(float, 32, false); }
        else { if (gather) LSTMSS_G1(float, 64, true); else LSTMSS_G1(float, 64, false); }
    }
#undef LSTMSS_G1
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
