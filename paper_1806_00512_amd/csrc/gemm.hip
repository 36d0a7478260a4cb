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

// --------------------------------------------------------------------------
// Data gradient: part[z][m][n] = sum over k in split z of W[row(k)][m] G[k][n]
// where row(k) = idx[k/P]*P + k%P (kept rows) or k (dense).
//
// Work-group tile TM x TN (4 wavefronts), K staged TK rows at a time through
// two LDS buffers: while the MFMAs consume one stage, the next stage's global
// loads are in flight in registers and are written to the other buffer, so a
// stage costs one barrier.  The gathered W row of every k of the split is
// looked up once into LDS.
//   fp32: LDS [k][m]; a lane's MFMA operand is one value, k = lane / 32.
//   bf16: the MFMA operand is 8 consecutive k of one row/column, so the
//         staging registers hold 4 k rows x VW columns and are transposed in
//         registers; LDS is [m][k] and a lane reads its operand as 16 bytes.
// --------------------------------------------------------------------------

template <typename TS, int TM, int TN>
struct G1Shape {
    static constexpr bool BF = sizeof(TS) == 2;
    static constexpr int TK = BF ? 64 : GEMM1_TK;   // k rows per stage
    static constexpr int KB = BF ? 4 : 1;           // k rows per staging group
    static constexpr int WM = TN == 32 ? 4 : 2;     // wavefront grid
    static constexpr int WN = 4 / WM;
    static constexpr int MT = TM / WM / 32, NT = TN / WN / 32;  // MFMA tiles per wavefront
    static constexpr int KSTEP = BF ? 16 : 2;       // k per MFMA
    static_assert(MT >= 1 && NT >= 1, "tile too small for four wavefronts");
};

template <typename TS, int TM, int TN, bool GATHER, bool VEC>
__global__ __launch_bounds__(THREADS) void gemm1_kernel(Gemm1Args a) {
    using SH = G1Shape<TS, TM, TN>;
    constexpr bool BF = SH::BF;
    constexpr int TK = SH::TK, KB = SH::KB, MT = SH::MT, NT = SH::NT, WM = SH::WM;
    using V = Vec<TS, VEC>;
    constexpr int VW = V::W;
    // staging groups (KB rows x VW columns) per stage and per thread
    constexpr int NA = (TK / KB) * (TM / VW), NB = (TK / KB) * (TN / VW);
    constexpr int RA = (NA + THREADS - 1) / THREADS, RB = (NB + THREADS - 1) / THREADS;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int mm0 = blockIdx.x * TM;
    const int n0 = blockIdx.y * TN;
    const int step = blockIdx.z / a.splitk, split = blockIdx.z - step * a.splitk;
    const int kb = split * (int)a.k_chunk;
    const int ke = min((int)a.Kp, kb + (int)a.k_chunk);
    const int M = a.M, N = a.N, ldw = (int)a.ldw;
    const TS *W = (const TS *)a.W;
    const TS *G = (const TS *)a.Gc + step * a.gc_step;
    const int32_t *idx = a.idx + (GATHER ? step * a.idx_step : 0);

    // gathered W row of every k of the current super-chunk (refilled every
    // GEMM1_KC_MAX rows; a multiple of TK)
    __shared__ int srow[GEMM1_KC_MAX];
    int sc = kb;
    auto fill_rows = [&](int s0) {
        const int s1 = min(ke, s0 + GEMM1_KC_MAX);
        for (int i = tid; i < s1 - s0; i += THREADS) {
            const int k = s0 + i;
            srow[i] = GATHER ? idx[k / a.P] * a.P + k % a.P : k;
        }
    };
    fill_rows(sc);

    // staging registers
    V ra[RA][KB], rb[RB][KB];
    auto load = [&](int k0) {
        int rows[RA][KB];
#pragma unroll
        for (int i = 0; i < RA; ++i)
#pragma unroll
            for (int r = 0; r < KB; ++r) {
                const int q = tid + i * THREADS;
                const int k = k0 + (q / (TM / VW)) * KB + r;
                rows[i][r] = q < NA && k < ke ? srow[k - sc] : -1;
            }
#pragma unroll
        for (int i = 0; i < RA; ++i) {
            const int q = tid + i * THREADS;
            const int m = a.m_lo + mm0 + (q % (TM / VW)) * VW;
#pragma unroll
            for (int r = 0; r < KB; ++r) {
                // a vector load never crosses the end of a W row: ldw is a
                // multiple of VW and so is m - m_lo; columns >= M are loaded
                // but never stored
                if (rows[i][r] >= 0 && m < M)
                    ra[i][r].load(W + (long)rows[i][r] * ldw + m, VW);
                else
                    ra[i][r].zero();
            }
        }
#pragma unroll
        for (int i = 0; i < RB; ++i) {
            const int q = tid + i * THREADS;
            const int n = n0 + (q % (TN / VW)) * VW;
#pragma unroll
            for (int r = 0; r < KB; ++r) {
                const int k = k0 + (q / (TN / VW)) * KB + r;
                if (q < NB && k < ke && n < N)
                    rb[i][r].load(G + (long)k * N + n, VW);
                else
                    rb[i][r].zero();
            }
        }
    };

    f32x16 acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                acc[i][j][v] = 0.f;
    const int mw = wm * MT * 32, nw = wn * NT * 32;  // wavefront tile origin

    if constexpr (!BF) {
        __shared__ __align__(16) float As[2][TK][TM + 4];
        __shared__ __align__(16) float Bs[2][TK][TN + 4];
        auto stash = [&](int buf) {
#pragma unroll
            for (int i = 0; i < RA; ++i) {
                const int q = tid + i * THREADS;
                if (q < NA) {
                    const int kk = q / (TM / VW), mm = (q % (TM / VW)) * VW;
#pragma unroll
                    for (int e = 0; e < VW; ++e)
                        As[buf][kk][mm + e] = ra[i][0].v[e];
                }
            }
#pragma unroll
            for (int i = 0; i < RB; ++i) {
                const int q = tid + i * THREADS;
                if (q < NB) {
                    const int kk = q / (TN / VW), nn = (q % (TN / VW)) * VW;
#pragma unroll
                    for (int e = 0; e < VW; ++e)
                        Bs[buf][kk][nn + e] = rb[i][0].v[e];
                }
            }
        };
        __syncthreads();
        load(kb);
        stash(0);
        __syncthreads();
        int buf = 0;
        for (int k0 = kb; k0 < ke; k0 += TK) {
            const bool next = k0 + TK < ke;
            if (next) {
                if (k0 + TK == sc + GEMM1_KC_MAX) {  // next super-chunk of rows
                    sc = k0 + TK;
                    fill_rows(sc);
                    __syncthreads();
                }
                load(k0 + TK);
            }
            float av[TK / 2][MT], bv[TK / 2][NT];
#pragma unroll
            for (int kk = 0; kk < TK / 2; ++kk) {
#pragma unroll
                for (int i = 0; i < MT; ++i)
                    av[kk][i] = As[buf][2 * kk + (lane >> 5)][mw + i * 32 + (lane & 31)];
#pragma unroll
                for (int j = 0; j < NT; ++j)
                    bv[kk][j] = Bs[buf][2 * kk + (lane >> 5)][nw + j * 32 + (lane & 31)];
            }
#pragma unroll
            for (int kk = 0; kk < TK / 2; ++kk)
#pragma unroll
                for (int i = 0; i < MT; ++i)
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        acc[i][j] = mfma32x32x2(av[kk][i], bv[kk][j], acc[i][j]);
            if (next)
                stash(buf ^ 1);
            __syncthreads();
            buf ^= 1;
        }
    } else {
        constexpr int LDK = TK + 8;  // row pitch 144 bytes: 16-byte reads of 32 rows spread over the banks
        __shared__ __align__(16) uint16_t As[2][TM][LDK];
        __shared__ __align__(16) uint16_t Bs[2][TN][LDK];
        // rows k0..k0+3 of column e packed as two dwords (k0 low)
        auto pack4 = [](const V *r, int e) {
            uint2 o;
            o.x = (uint32_t)r[0].v[e] | ((uint32_t)r[1].v[e] << 16);
            o.y = (uint32_t)r[2].v[e] | ((uint32_t)r[3].v[e] << 16);
            return o;
        };
        auto stash = [&](int buf) {
#pragma unroll
            for (int i = 0; i < RA; ++i) {
                const int q = tid + i * THREADS;
                if (q < NA) {
                    const int kk = (q / (TM / VW)) * KB, mm = (q % (TM / VW)) * VW;
#pragma unroll
                    for (int e = 0; e < VW; ++e)
                        *(uint2 *)&As[buf][mm + e][kk] = pack4(ra[i], e);
                }
            }
#pragma unroll
            for (int i = 0; i < RB; ++i) {
                const int q = tid + i * THREADS;
                if (q < NB) {
                    const int kk = (q / (TN / VW)) * KB, nn = (q % (TN / VW)) * VW;
#pragma unroll
                    for (int e = 0; e < VW; ++e)
                        *(uint2 *)&Bs[buf][nn + e][kk] = pack4(rb[i], e);
                }
            }
        };
        __syncthreads();
        load(kb);
        stash(0);
        __syncthreads();
        int buf = 0;
        for (int k0 = kb; k0 < ke; k0 += TK) {
            const bool next = k0 + TK < ke;
            if (next) {
                if (k0 + TK == sc + GEMM1_KC_MAX) {
                    sc = k0 + TK;
                    fill_rows(sc);
                    __syncthreads();
                }
                load(k0 + TK);
            }
            u16x8 av[TK / 16][MT], bv[TK / 16][NT];
#pragma unroll
            for (int kk = 0; kk < TK / 16; ++kk) {
#pragma unroll
                for (int i = 0; i < MT; ++i)
                    av[kk][i] = *(const u16x8 *)&As[buf][mw + i * 32 + (lane & 31)][16 * kk + 8 * (lane >> 5)];
#pragma unroll
                for (int j = 0; j < NT; ++j)
                    bv[kk][j] = *(const u16x8 *)&Bs[buf][nw + j * 32 + (lane & 31)][16 * kk + 8 * (lane >> 5)];
            }
#pragma unroll
            for (int kk = 0; kk < TK / 16; ++kk)
#pragma unroll
                for (int i = 0; i < MT; ++i)
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        acc[i][j] = mfma32x32x16bf(av[kk][i], bv[kk][j], acc[i][j]);
            if (next)
                stash(buf ^ 1);
            __syncthreads();
            buf ^= 1;
        }
    }

    float *out = a.part + step * a.out_step + split * a.part_stride;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const int n = n0 + nw + j * 32 + (lane & 31);
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = a.m_lo + mm0 + mw + i * 32 + acc_row(lane, v);
                if (m >= a.m_begin && m < M && n < N)
                    out[(long)(m - a.out_row0) * N + n] = acc[i][j][v];
            }
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
// Weight gradient of all time steps in one launch.
//
// Work-group: one group of output rows x 128 features (4 waves x 32).  It
// walks the launch's time steps (and batch chunks) and owns its dW tile, so
// dW is written (or, for a later chunk of steps, updated) once per launch in
// a fixed summation order (deterministic, no atomics).
//
// Dense: a group is 32 consecutive rows; each step's product is added to the
// accumulator.
// Sparse: a group is `greg` consecutive regions.  Every full region keeps
// exactly (R-S)*P rows, so at every step the group's kept rows are the same
// contiguous range of compacted rows (at most 32*TT of them).  The MFMA
// accumulates those into a temporary tile whose columns are kept rows; after
// the step each accumulator column (an original row) pulls its value from the
// temporary column holding it (ds_bpermute across lanes of the same half),
// or nothing if its slice was dropped at that step.  The MFMA work is thus
// only the kept rows' (no zero-filled rows).
//
// MFMA operands: A = [x_t; h_{t-1}] rows (features), B = gate-gradient rows;
// accumulator column = row of dW (lane), accumulator rows = features.  Lanes
// 0-31 consume batch columns [0, BC/2) of the chunk and lanes 32-63
// [BC/2, BC), so each lane reads consecutive columns from LDS.
// --------------------------------------------------------------------------
constexpr int WG_FEAT = 128;
constexpr int WG_ATMAX = 4;

constexpr int WG_NG = 2;   // row groups per work-group
constexpr int WG_FT = 2;   // 32-feature tiles per wavefront

// Stores a staged vector into an LDS row (one 16-byte store when whole).
template <typename E, typename V>
__device__ __forceinline__ void lds_store_vec(E *dst, const V &v) {
    if constexpr (V::W * sizeof(E) == 16) {
        typedef E e16 __attribute__((ext_vector_type(16 / sizeof(E))));
        e16 t;
#pragma unroll
        for (int e = 0; e < V::W; ++e)
            t[e] = v.v[e];
        *(e16 *)dst = t;
    } else {
#pragma unroll
        for (int e = 0; e < V::W; ++e)
            dst[e] = v.v[e];
    }
}

template <typename TS, bool SPARSE, int TT, int ATN, bool VEC, int BC>
__global__ __launch_bounds__(THREADS, 2) void wgrad_kernel(WgradArgs a) {
    using E = typename std::conditional<sizeof(TS) == 4, float, uint16_t>::type;
    constexpr int PITCH = BC + (sizeof(TS) == 4 ? 4 : 8);
    constexpr int GROWS = TT * 32;                // temporary-tile rows per group
    using V = Vec<TS, VEC>;
    constexpr int VW = V::W;
    constexpr int cpr = BC / VW;
    constexpr int gvec = WG_NG * GROWS * cpr, xvec = WG_FEAT * cpr;
    constexpr int RG = (gvec + THREADS - 1) / THREADS;
    constexpr int RX = (xvec + THREADS - 1) / THREADS;
    __shared__ __align__(16) E sX[WG_FEAT][PITCH];
    __shared__ __align__(16) E sG[WG_NG * GROWS][PITCH];
    __shared__ int sidx[WG_NG][64];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int fh = wave & 1, gi = wave >> 1;      // feature half, group of this wavefront
    const int I = a.I, H = a.H, B = a.B;
    const int NC = I + H, G4 = 4 * H;
    const int n0 = blockIdx.y * WG_FEAT;
    const TS *Gc = (const TS *)a.Gc;
    const TS *x = (const TS *)a.x;
    const TS *h = (const TS *)a.h;

    // geometry of group g: original rows [r0, r0 + rcount), compacted rows
    // [c0, c0 + ccount), kept-slice entries [q0, q0 + qcount), first slice j0
    const int rp = a.R * a.P, kr = (a.R - a.S) * a.P, ks = a.R - a.S;
    auto geom = [&](int g, int &r0, int &rcount, int &c0, int &ccount, int &q0, int &qcount,
                    int &j0) {
        if (SPARSE) {
            r0 = g * a.greg * rp;
            rcount = max(0, min(a.greg * rp, G4 - r0));
            c0 = g * a.greg * kr;
            ccount = max(0, min(a.greg * kr, a.Kp - c0));
            q0 = g * a.greg * ks;
            qcount = max(0, min(a.greg * ks, a.kept - q0));
            j0 = g * a.greg * a.R;
        } else {
            r0 = g * 32;
            rcount = max(0, min(32, G4 - r0));
            c0 = r0;
            ccount = rcount;
            q0 = qcount = j0 = 0;
        }
    };
    int r0, rcount, c0, ccount, q0, qcount, j0;
    geom(blockIdx.x * WG_NG + gi, r0, rcount, c0, ccount, q0, qcount, j0);
    const int AT = SPARSE ? (rcount + 31) / 32 : 1;
    // compacted-row origin and count of both groups, for the loaders
    int lc0[WG_NG], lcc[WG_NG], lq0[WG_NG], lqc[WG_NG];
#pragma unroll
    for (int k = 0; k < WG_NG; ++k) {
        int t0, t1, t2, t3;
        geom(blockIdx.x * WG_NG + k, t0, t1, lc0[k], lcc[k], lq0[k], lqc[k], t2);
        (void)t3;
    }

    const int nbc = (B + BC - 1) / BC;
    const int niters = (a.t_end - a.t_begin) * nbc;

    V rg[RG], rx[RX];
    int ridx = -1;
    auto load = [&](int it) {
        const int tl = it / nbc, b0 = (it - tl * nbc) * BC;
        const int t = a.t_begin + tl;
        const TS *Gt = Gc + (long)t * a.Kp * B;
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const int q = tid + i * THREADS;
            const int rho = q / cpr, bb = (q - rho * cpr) * VW;
            const int k = rho / GROWS, lr = rho - k * GROWS;
            const int b = b0 + bb;
            if (q < gvec && lr < lcc[k & (WG_NG - 1)] && b < B)
                rg[i].load(Gt + (long)(lc0[k & (WG_NG - 1)] + lr) * B + b, B - b);
            else
                rg[i].zero();
        }
#pragma unroll
        for (int i = 0; i < RX; ++i) {
            const int q = tid + i * THREADS;
            const int f = q / cpr, bb = (q - f * cpr) * VW;
            const int n = n0 + f, b = b0 + bb;
            if (q < xvec && n < NC && b < B) {
                const TS *src = n < I ? x + ((long)t * I + n) * B : h + ((long)t * H + (n - I)) * B;
                rx[i].load(src + b, B - b);
            } else {
                rx[i].zero();
            }
        }
        if (SPARSE && b0 == 0 && tid < WG_NG * 64) {
            const int k = tid >> 6, e = tid & 63;
            ridx = e < lqc[k] ? a.idx[(long)t * a.kept + lq0[k] + e] : -1;
        }
    };

    f32x16 acc[WG_FT][ATN], tmp[WG_FT][TT];
#pragma unroll
    for (int ft = 0; ft < WG_FT; ++ft) {
#pragma unroll
        for (int j = 0; j < ATN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                acc[ft][j][v] = 0.f;
#pragma unroll
        for (int j = 0; j < TT; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                tmp[ft][j][v] = 0.f;
    }

    load(0);
    constexpr int HALF = BC / 2;
    const int hb = (lane >> 5) * HALF;
    for (int it = 0; it < niters; ++it) {
        const int bc = it % nbc;
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const int q = tid + i * THREADS;
            if (q < gvec) {
                const int rho = q / cpr, bb = (q - rho * cpr) * VW;
                lds_store_vec(&sG[rho][bb], rg[i]);
            }
        }
#pragma unroll
        for (int i = 0; i < RX; ++i) {
            const int q = tid + i * THREADS;
            if (q < xvec) {
                const int f = q / cpr, bb = (q - f * cpr) * VW;
                lds_store_vec(&sX[f][bb], rx[i]);
            }
        }
        if (SPARSE && bc == 0 && tid < WG_NG * 64)
            sidx[tid >> 6][tid & 63] = ridx;
        __syncthreads();
        if (it + 1 < niters)
            load(it + 1);

        // MFMA over this batch chunk: 2 feature tiles x TT row tiles
        if constexpr (sizeof(TS) == 4) {
#pragma unroll 2
            for (int s4 = 0; s4 < HALF; s4 += 4) {
                float4 av[WG_FT], bv[TT];
#pragma unroll
                for (int ft = 0; ft < WG_FT; ++ft)
                    av[ft] = *(const float4 *)&sX[fh * 64 + ft * 32 + (lane & 31)][hb + s4];
#pragma unroll
                for (int tt = 0; tt < TT; ++tt)
                    bv[tt] = *(const float4 *)&sG[gi * GROWS + tt * 32 + (lane & 31)][hb + s4];
#pragma unroll
                for (int ft = 0; ft < WG_FT; ++ft)
#pragma unroll
                    for (int tt = 0; tt < TT; ++tt) {
                        f32x16 &c = tmp[ft][tt];
                        c = mfma32x32x2(av[ft].x, bv[tt].x, c);
                        c = mfma32x32x2(av[ft].y, bv[tt].y, c);
                        c = mfma32x32x2(av[ft].z, bv[tt].z, c);
                        c = mfma32x32x2(av[ft].w, bv[tt].w, c);
                    }
            }
        } else {
#pragma unroll 2
            for (int s8 = 0; s8 < HALF; s8 += 8) {
                u16x8 av[WG_FT], bv[TT];
#pragma unroll
                for (int ft = 0; ft < WG_FT; ++ft)
                    av[ft] = *(const u16x8 *)&sX[fh * 64 + ft * 32 + (lane & 31)][hb + s8];
#pragma unroll
                for (int tt = 0; tt < TT; ++tt)
                    bv[tt] = *(const u16x8 *)&sG[gi * GROWS + tt * 32 + (lane & 31)][hb + s8];
#pragma unroll
                for (int ft = 0; ft < WG_FT; ++ft)
#pragma unroll
                    for (int tt = 0; tt < TT; ++tt)
                        tmp[ft][tt] = mfma32x32x16bf(av[ft], bv[tt], tmp[ft][tt]);
            }
        }

        // end of a step: dense adds the step's product; sparse routes each
        // kept row of the step into its original row (same summation order
        // either way, so a sparse call that keeps every row matches the
        // dense one bit for bit)
        if (bc == nbc - 1) {
            if (!SPARSE) {
#pragma unroll
                for (int ft = 0; ft < WG_FT; ++ft)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        acc[ft][0][v] += tmp[ft][0][v];
                        tmp[ft][0][v] = 0.f;
                    }
            } else {
#pragma unroll
                for (int at = 0; at < ATN; ++at) {
                    if (at >= AT)
                        break;
                    const int col = at * 32 + (lane & 31);
                    int src = -1;
                    if (col < rcount) {
                        const int orow = r0 + col;
                        const int js = orow / a.P;
                        const int reg = (js - j0) / a.R;
                        const int e0 = reg * ks, e1 = min(e0 + ks, qcount);
                        for (int e = e0; e < e1; ++e)
                            if (sidx[gi][e] == js)
                                src = e * a.P + (orow - js * a.P);
                    }
                    const int saddr = (((src < 0 ? 0 : src) & 31) + (lane & 32)) << 2;
                    const int stile = src < 0 ? 0 : (src >> 5);
#pragma unroll
                    for (int ft = 0; ft < WG_FT; ++ft)
#pragma unroll
                        for (int v = 0; v < 16; ++v) {
                            float val = __int_as_float(
                                __builtin_amdgcn_ds_bpermute(saddr, __float_as_int(tmp[ft][0][v])));
                            if (TT > 1) {
                                const float v1 = __int_as_float(__builtin_amdgcn_ds_bpermute(
                                    saddr, __float_as_int(tmp[ft][TT > 1 ? 1 : 0][v])));
                                val = stile == 1 ? v1 : val;
                            }
                            acc[ft][at][v] += src < 0 ? 0.f : val;
                        }
                }
#pragma unroll
                for (int ft = 0; ft < WG_FT; ++ft)
#pragma unroll
                    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                        for (int v = 0; v < 16; ++v)
                            tmp[ft][tt][v] = 0.f;
            }
        }
        __syncthreads();
    }

    // write the owned tile of dW
#pragma unroll
    for (int at = 0; at < ATN; ++at) {
        if (at >= AT)
            break;
        const int col = at * 32 + (lane & 31);
        if (col >= rcount)
            continue;
        float *dst = a.dW + (long)(r0 + col) * NC;
#pragma unroll
        for (int ft = 0; ft < WG_FT; ++ft)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int f = n0 + fh * 64 + ft * 32 + acc_row(lane, v);
                if (f < NC)
                    dst[f] = a.accumulate ? dst[f] + acc[ft][at][v] : acc[ft][at][v];
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

// Tile of the data-gradient GEMM.  Its operands stream from L2 / MALL, so
// occupancy beats operand reuse: fp32 runs 64 x 64 tiles (three work-groups
// per CU); bf16, whose MFMA is 8x faster per byte staged, runs 128 x 128.
void gemm1_tile(bool bf16, int N, int *tm, int *tn) {
    if (N <= 32) {
        *tm = 128;
        *tn = 32;
    } else if (!bf16 || N <= 64) {
        *tm = bf16 ? 128 : 64;
        *tn = 64;
    } else {
        *tm = 128;
        *tn = 128;
    }
}

hipError_t launch_gemm1(Gemm1Args a, bool bf16, hipStream_t s) {
    if (a.k_chunk % GEMM1_TK != 0 || a.splitk < 1 || a.steps < 1)
        return hipErrorInvalidValue;
    // 16-byte vector loads need 16-byte aligned rows; the tile origin is
    // rounded down to the vector width and rows below m_begin are not stored
    const int vw = bf16 ? 8 : 4;
    const bool vec = a.ldw % vw == 0 && a.N % vw == 0;
    a.m_lo = vec ? a.m_begin / vw * vw : a.m_begin;
    const long z = (long)a.splitk * a.steps;
    int TM, TN;
    gemm1_tile(bf16, a.N, &TM, &TN);
    if (a.tm)
        TM = a.tm;
    if (a.tn)
        TN = a.tn;
    if (!((TN == 32 && TM == 128) || ((TN == 64 || TN == 128) && (TM == 64 || TM == 128))))
        return hipErrorInvalidValue;
    dim3 grid((unsigned)ceil_div(a.M - a.m_lo, TM), (unsigned)ceil_div(a.N, TN), (unsigned)z);
    const bool gather = a.idx != nullptr;
#define LSTMSS_G1(TS, TMV, TNV, GA, VE) hipLaunchKernelGGL((gemm1_kernel<TS, TMV, TNV, GA, VE>), grid, dim3(THREADS), 0, s, a)
#define LSTMSS_G1V(TS, TMV, TNV, GA) do { if (vec) LSTMSS_G1(TS, TMV, TNV, GA, true); else LSTMSS_G1(TS, TMV, TNV, GA, false); } while (0)
#define LSTMSS_G1T(TS, GA) do { \
        if (TN == 32) LSTMSS_G1V(TS, 128, 32, GA); \
        else if (TN == 64) { if (TM == 128) LSTMSS_G1V(TS, 128, 64, GA); else LSTMSS_G1V(TS, 64, 64, GA); } \
        else { if (TM == 128) LSTMSS_G1V(TS, 128, 128, GA); else LSTMSS_G1V(TS, 64, 128, GA); } } while (0)
    if (bf16) { if (gather) LSTMSS_G1T(bf16_t, true); else LSTMSS_G1T(bf16_t, false); }
    else { if (gather) LSTMSS_G1T(float, true); else LSTMSS_G1T(float, false); }
#undef LSTMSS_G1T
#undef LSTMSS_G1V
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

// Temporary tiles (kept rows per group / 32) and accumulator tiles (original
// rows per group / 32) of the sparse weight-gradient kernel.
static void wgrad_tiles(int P, int R, int S, int *greg, int *tt, int *at) {
    const int kr = (R - S) * P, rp = R * P;
    *greg = kr <= 32 ? max(1, 32 / kr) : 1;
    *tt = (*greg * kr + 31) / 32;
    *at = (*greg * rp + 31) / 32;
}

bool wgrad_supported(int P, int R, int S) {
    int greg, tt, at;
    wgrad_tiles(P, R, S, &greg, &tt, &at);
    return tt <= 2 && at <= WG_ATMAX && (R - S) <= 64;
}

hipError_t launch_wgrad(WgradArgs a, bool sparse, bool bf16, hipStream_t s) {
    int tt = 1, at = 1;
    if (sparse) {
        if (!wgrad_supported(a.P, a.R, a.S))
            return hipErrorNotSupported;
        wgrad_tiles(a.P, a.R, a.S, &a.greg, &tt, &at);
    }
    // batch columns per stage: 16/32 (fp32) or 32/64 (bf16, whole MFMA
    // k-blocks); larger stages would not leave room for two wavefronts per SIMD
    int bc = a.B <= 16 ? 16 : a.B <= 32 ? 32 : (bf16 ? 64 : 32);
    a.BC = bc;
    const int vw = bf16 ? 8 : 4;
    const bool vec = a.B % vw == 0;
    const long groups = sparse ? ceil_div(ceil_div(4L * a.H / a.P, a.R), a.greg) : ceil_div(4L * a.H, 32);
    dim3 grid((unsigned)ceil_div(groups, WG_NG), (unsigned)ceil_div(a.I + a.H, WG_FEAT));
#define LSTMSS_WG(TS, SP, TTV, ATV, VE) do { \
        if (bc == 16) hipLaunchKernelGGL((wgrad_kernel<TS, SP, TTV, ATV, VE, 16>), grid, dim3(THREADS), 0, s, a); \
        else if (bc == 32) hipLaunchKernelGGL((wgrad_kernel<TS, SP, TTV, ATV, VE, 32>), grid, dim3(THREADS), 0, s, a); \
        else hipLaunchKernelGGL((wgrad_kernel<TS, SP, TTV, ATV, VE, 64>), grid, dim3(THREADS), 0, s, a); } while (0)
#define LSTMSS_WGV(TS, SP, TTV, ATV) do { if (vec) LSTMSS_WG(TS, SP, TTV, ATV, true); else LSTMSS_WG(TS, SP, TTV, ATV, false); } while (0)
#define LSTMSS_WGA(TS, TTV) do { \
        if (at <= 1) LSTMSS_WGV(TS, true, TTV, 1); else if (at <= 2) LSTMSS_WGV(TS, true, TTV, 2); \
        else LSTMSS_WGV(TS, true, TTV, 4); } while (0)
    if (bf16) {
        if (!sparse) LSTMSS_WGV(bf16_t, false, 1, 1);
        else if (tt == 1) LSTMSS_WGA(bf16_t, 1);
        else LSTMSS_WGA(bf16_t, 2);
    } else {
        if (!sparse) LSTMSS_WGV(float, false, 1, 1);
        else if (tt == 1) LSTMSS_WGA(float, 1);
        else LSTMSS_WGA(float, 2);
    }
#undef LSTMSS_WGA
#undef LSTMSS_WGV
#undef LSTMSS_WG
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
