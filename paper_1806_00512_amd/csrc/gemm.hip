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
//
// Both operands arrive k-major (W rows, gate-gradient rows) while an MFMA
// operand is a run of consecutive k of one row/column, so a thread stages 4 k
// rows x VW columns, transposes them in registers and stores each column's 4
// k values as one vector; LDS is [m][k] and a lane reads 4 (fp32) or 8
// (bf16) consecutive k with one 16-byte read.  fp32 MFMA c of an 8-k block
// contracts k = 8b + c (lanes 0-31) and k = 8b + 4 + c (lanes 32-63), the
// same for both operands.
// --------------------------------------------------------------------------

template <typename TS, int TM, int TN, int NW = 4>
struct G1Shape {
    static constexpr bool BF = sizeof(TS) == 2;
    static constexpr int TK = BF ? 64 : 32;         // k rows per stage
    static constexpr int KB = 4;                    // k rows per staging group
    static constexpr int WM = NW == 8 ? 4 : (TN == 32 ? 4 : 2);  // wavefront grid
    static constexpr int WN = NW / WM;
    static constexpr int MT = TM / WM / 32, NT = TN / WN / 32;  // MFMA tiles per wavefront
    static constexpr int LDK = TK + (BF ? 8 : 4);   // LDS row pitch (144 bytes)
    static_assert(MT >= 1 && NT >= 1, "tile too small for its wavefronts");
    static_assert(GEMM1_TK % TK == 0 && GEMM1_KC_MAX % TK == 0, "stage must divide the split granularity");
};

// ROWA: the forward products a = W[:, kcol0 : kcol0 + Kp] G instead, whose
// first operand arrives row-major with k contiguous: a thread stages KB rows
// x VW consecutive k and stores each row's vector as it is.
// FN: the fine structure with 32-row slices and 32-column blocks on the
// masked matrix, with TN = 32 (a work-group's columns are one block): the
// work-group gathers the rows of the slices that keep its block and skips
// the others, W rows and gate-gradient rows alike (their products are exactly
// zero, so the result is bit-identical to multiplying them).
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glob_void_t;

// DMA (whole k stages): the stages go from global memory straight into LDS
// (global_load_lds_dwordx4) in the operands' own layout, [k][m] and [k][n]
// with m, n contiguous, instead of being transposed through registers.
//   fp32: a lane reads its one k of each MFMA operand with a 4-byte read; the
//   128-byte halves of every row are swapped in alternate groups of 4 rows (k
//   and k + 4 are read together).
//   bf16 (128 x 128 tiles, eight wavefronts): a lane needs 8 consecutive k of
//   one column, which two transposed reads (ds_read_b64_tr_b16) deliver: in
//   each group of 16 lanes, lane s points at row kbase + s / 4, columns
//   mbase + 4 (s % 4) .. + 3, and lane i receives rows kbase .. kbase + 3 of
//   column mbase + i.  Row r's 16-byte pieces are permuted by g1_swz16(r), so
//   that the 4 rows x 2 pieces a group reads, and the 16 pieces two groups
//   read together, fall on distinct banks.
// The permutations are applied on the global side of the copy.  Columns past
// M or N are clamped to the last whole piece of the row (their outputs are
// not stored).
__device__ __forceinline__ int g1_swz(int k) { return ((k >> 2) & 1) * 8; }  // in 16-byte pieces
__device__ __forceinline__ int g1_swz16(int k) { return ((k & 3) << 2) ^ (((k >> 1) & 1) << 1); }
// ROWA (forward products): the first operand's rows are k-contiguous 128-byte
// lines ([m][k], TK elements), read 16 bytes at a time like the weight
// gradient's; piece c of row r sits at c ^ g1_swzr(r).
__device__ __forceinline__ int g1_swzr(int r) { return (r & 7) ^ ((r >> 3) & 1); }
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 g1_bf16x4;
typedef __attribute__((address_space(3))) g1_bf16x4 g1_lds_bf16x4;
typedef short g1_s16x4 __attribute__((ext_vector_type(4)));

template <typename TS, int TM, int TN, bool GATHER, bool VEC, bool ROWA = false, int NW = 4,
          bool FN = false, bool DMA = false>
__global__ __launch_bounds__(NW * 64) void gemm1_kernel(Gemm1Args a) {
    static_assert(!(ROWA && GATHER), "the forward products read every row");
    static_assert(!(FN && (GATHER || ROWA)), "the fine fast path reads every row");
    static_assert(!DMA || (!FN && VEC &&
                           (sizeof(TS) == 4 ? NW == 4 : (NW == 8 && TM == 128 && TN == 128))),
                  "DMA stages: fp32 products, or bf16 128 x 128 tiles of eight wavefronts");
    constexpr int THREADS = NW * 64;  // shadows the file-wide default
    using SH = G1Shape<TS, TM, TN, NW>;
    constexpr bool BF = SH::BF;
    constexpr int TK = SH::TK, KB = SH::KB, MT = SH::MT, NT = SH::NT, WM = SH::WM, LDK = SH::LDK;
    using E = typename std::conditional<BF, uint16_t, float>::type;
    using V = Vec<TS, VEC>;
    constexpr int VW = V::W;
    // staging groups (KB rows x VW columns) per stage; when both operands'
    // groups fit one pass, threads [0, NA) stage W and [NA, NA + NB) stage G.
    // Consecutive threads take consecutive k groups of one column block: 8
    // (fp32) or 16 (bf16) lanes then store into distinct LDS banks, and each
    // row segment they load is 128 contiguous bytes
    constexpr int NA = (TK / KB) * (TM / VW), NB = (TK / KB) * (TN / VW);
    constexpr bool SPLIT = NA + NB <= THREADS;
    constexpr int RA = SPLIT ? 1 : (NA + THREADS - 1) / THREADS;
    constexpr int RB = SPLIT ? 1 : (NB + THREADS - 1) / THREADS;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int mm0 = blockIdx.x * TM;
    const int n0 = blockIdx.y * TN;
    const int step = blockIdx.z / a.splitk, split = blockIdx.z - step * a.splitk;
    const int kb = split * (int)a.k_chunk;
    const int ke0 = min((int)a.Kp, kb + (int)a.k_chunk);
    const int M = a.M, N = a.N, ldw = (int)a.ldw;
    const TS *W = (const TS *)a.W;
    const TS *G = (const TS *)a.Gc + step * a.gc_step;
    const int32_t *idx = a.idx + (GATHER ? step * a.idx_step : 0);

    // FN: slices of [kb, ke0) that keep this work-group's column block, in
    // ascending order (one wavefront compacts them with ballots)
    __shared__ int slist[FN ? FINE_MAX_SLICES : 1];
    __shared__ int s_nact;
    int ke = ke0;
    if constexpr (FN) {
        static_assert(!FN || TN == 32, "a fine work-group's columns are one block");
        if (tid < 64) {
            const int32_t *fi = a.fidx + step * a.fidx_step;
            const int c = n0 >> 5, s_end = ke0 >> 5;
            int base = 0;
            for (int sb = kb >> 5; sb < s_end; sb += 64) {
                const int sl = sb + tid;
                bool kept = false;
                if (sl < s_end) {
                    const int32_t *e = fi + (long)sl * a.fkept;
                    for (int q = 0; q < a.fkept; ++q)
                        kept |= e[q] == c;
                }
                const uint64_t m = __ballot(kept);
                if (kept)
                    slist[base + __popcll(m & ((1ull << tid) - 1ull))] = sl;
                base += __popcll(m);
            }
            if (tid == 0)
                s_nact = base;
        }
        __syncthreads();
        ke = kb + s_nact * 32;
    }
    // gate-gradient row of compacted position k (FN), else k itself
    auto grow = [&](int k) { return FN ? slist[(k - kb) >> 5] * 32 + ((k - kb) & 31) : k; };

    // gathered W row of every k of the current super-chunk (refilled every
    // GEMM1_KC_MAX rows, a multiple of TK)
    __shared__ int srow[GEMM1_KC_MAX];
    int sc = kb;
    auto fill_rows = [&](int s0) {
        const int s1 = min(ke, s0 + GEMM1_KC_MAX);
        for (int i = tid; i < s1 - s0; i += THREADS) {
            const int k = s0 + i;
            srow[i] = GATHER ? idx[k / a.P] * a.P + k % a.P : k;
        }
    };
    if (!ROWA && !FN)
        fill_rows(sc);

    auto qa = [&](int i) { return tid + i * THREADS; };
    auto qb = [&](int i) { return SPLIT ? tid - NA : tid + i * THREADS; };
    V ra[RA][KB], rb[RB][KB];
    auto load = [&](int k0) {
#pragma unroll
        for (int i = 0; i < RA; ++i) {
            const int q = qa(i);
            if constexpr (ROWA) {
                // KB rows m x VW consecutive k; kcol0 and ldw are multiples
                // of VW when VEC, so a vector never crosses a row or ke
                const int k = k0 + (q % (TK / VW)) * VW;
                const int m = mm0 + (q / (TK / VW)) * KB;
#pragma unroll
                for (int r = 0; r < KB; ++r) {
                    if (q < NA && m + r < M && k < ke)
                        ra[i][r].load(W + (long)(m + r) * ldw + a.kcol0 + k, ke - k);
                    else
                        ra[i][r].zero();
                }
                continue;
            }
            const int kg = k0 + (q % (TK / KB)) * KB;
            const int m = a.m_lo + mm0 + (q / (TK / KB)) * VW;
            // a vector load never crosses the end of a W row: ldw is a
            // multiple of VW and so is m - m_lo; columns >= M are loaded but
            // never stored
            const bool ok = q < NA && m < M;
#pragma unroll
            for (int r = 0; r < KB; ++r) {
                const int k = kg + r;
                if (ok && k < ke)
                    ra[i][r].load(W + (long)(FN ? grow(k) : srow[k - sc]) * ldw + m, VW);
                else
                    ra[i][r].zero();
            }
        }
#pragma unroll
        for (int i = 0; i < RB; ++i) {
            const int q = qb(i);
            const int kg = k0 + (q % (TK / KB)) * KB;
            const int n = n0 + (q / (TK / KB)) * VW;
            const bool ok = q >= 0 && q < NB && n < N;
#pragma unroll
            for (int r = 0; r < KB; ++r) {
                const int k = kg + r;
                if (ok && k < ke)
                    rb[i][r].load(G + (long)grow(k) * N + n, VW);
                else
                    rb[i][r].zero();
            }
        }
    };

    __shared__ __align__(16) E As[2][DMA ? 1 : TM][LDK];
    __shared__ __align__(16) E Bs[2][DMA ? 1 : TN][LDK];
    __shared__ __align__(16) E Ad[2][DMA ? TK * TM : 1];  // DMA: [k][m]
    __shared__ __align__(16) E Bd[2][DMA ? TK * TN : 1];  // DMA: [k][n]
    // DMA copy of the stage starting at k0 into buffer b: instruction q fills
    // bytes [1024 q, 1024 q + 1024) of Ad (q < NIA) or of Bd
    constexpr int PEL = 16 / (int)sizeof(E), IEL = 1024 / (int)sizeof(E);  // elements per piece / instruction
    constexpr int NIA = TK * TM / IEL, NIB = TK * TN / IEL, NIW = (NIA + NIB) / NW;
    static_assert(!DMA || (NIA + NIB) % NW == 0, "DMA instruction split");
    auto swz = [](int k) { return BF ? g1_swz16(k) : g1_swz(k); };
    auto dload = [&](int k0, int b) {
#pragma unroll
        for (int i = 0; i < NIW; ++i) {
            const int q = wave + NW * i;
            const bool isa = q < NIA;
            const int off = (isa ? q : q - NIA) * IEL + lane * PEL;  // element offset in the stage
            const int rowlen = isa ? TM : TN;
            const int kl = off / rowlen, pc = (off - kl * rowlen) / PEL;
            const int col = (pc ^ swz(kl)) * PEL;  // first column this lane's slot holds
            const TS *src;
            if (isa && ROWA) {
                // row kl' = off / TK of the [m][k] tile, piece pc' of it
                const int ml = off / TK, pr = (off - ml * TK) / PEL;
                const int m = min(mm0 + ml, M - 1);
                src = W + (long)m * ldw + a.kcol0 + k0 + (pr ^ g1_swzr(ml)) * PEL;
            } else if (isa) {
                const int m = min(a.m_lo + mm0 + col, ((M - 1) & ~(PEL - 1)));
                src = W + (long)srow[k0 + kl - sc] * ldw + m;
            } else {
                const int n = min(n0 + col, N - PEL);
                src = G + (long)(k0 + kl) * N + n;
            }
            E *dst = isa ? &Ad[b][q * IEL] : &Bd[b][(q - NIA) * IEL];
            __builtin_amdgcn_global_load_lds((glob_void_t *)src, (lds_void_t *)dst, 16, 0, 0);
        }
    };
    // column e of a group: its KB = 4 k values as one vector (k lowest first)
    auto put4 = [](E *dst, const V *r, int e) {
        if constexpr (BF) {
            uint2 o;
            o.x = (uint32_t)r[0].v[e] | ((uint32_t)r[1].v[e] << 16);
            o.y = (uint32_t)r[2].v[e] | ((uint32_t)r[3].v[e] << 16);
            *(uint2 *)dst = o;
        } else {
            *(float4 *)dst = make_float4(r[0].v[e], r[1].v[e], r[2].v[e], r[3].v[e]);
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int i = 0; i < RA; ++i) {
            const int q = qa(i);
            if (ROWA && q < NA) {
                const int kk = (q % (TK / VW)) * VW, mm = (q / (TK / VW)) * KB;
#pragma unroll
                for (int r = 0; r < KB; ++r) {
                    E *dst = &As[buf][mm + r][kk];
                    if constexpr (VW == 1) {
                        *dst = ra[i][r].v[0];
                    } else if constexpr (BF) {
                        u16x8 t;
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            t[e] = ra[i][r].v[e];
                        *(u16x8 *)dst = t;
                    } else {
                        *(float4 *)dst = make_float4(ra[i][r].v[0], ra[i][r].v[1], ra[i][r].v[2],
                                                     ra[i][r].v[3]);
                    }
                }
            } else if (q < NA) {
                const int kk = (q % (TK / KB)) * KB, mm = (q / (TK / KB)) * VW;
#pragma unroll
                for (int e = 0; e < VW; ++e)
                    put4(&As[buf][mm + e][kk], ra[i], e);
            }
        }
#pragma unroll
        for (int i = 0; i < RB; ++i) {
            const int q = qb(i);
            if (q >= 0 && q < NB) {
                const int kk = (q % (TK / KB)) * KB, nn = (q / (TK / KB)) * VW;
#pragma unroll
                for (int e = 0; e < VW; ++e)
                    put4(&Bs[buf][nn + e][kk], rb[i], e);
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

    __syncthreads();
    if constexpr (DMA) {
        dload(kb, 0);
        __builtin_amdgcn_s_waitcnt(0);
    } else {
        load(kb);
        stash(0);
    }
    __syncthreads();
    int buf = 0;
    for (int k0 = kb; k0 < ke; k0 += TK) {
        const bool next = k0 + TK < ke;
        if (next) {
            if (!ROWA && !FN && k0 + TK == sc + GEMM1_KC_MAX) {  // next super-chunk of rows
                sc = k0 + TK;
                fill_rows(sc);
                __syncthreads();
            }
            if (!DMA)
                load(k0 + TK);
        }
        const int half = lane >> 5;
        if constexpr (DMA && BF) {
            // two transposed reads per operand and 16-k block: rows
            // 16 kk + 8 half + 4 h + (0..3) of column (lane % 32)
            const int g = lane >> 4, sl = lane & 15;
            auto trd = [](const E *p) {
                return __builtin_bit_cast(
                    g1_s16x4, __builtin_amdgcn_ds_read_tr16_b64_v4bf16((g1_lds_bf16x4 *)(p)));
            };
            u16x8 av[TK / 16][MT], bv[TK / 16][NT];
#pragma unroll
            for (int kk = 0; kk < TK / 16; ++kk) {
                g1_s16x4 ra[2][MT], rb[2][NT];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int k = 16 * kk + 8 * (g >> 1) + 4 * h + (sl >> 2);
#pragma unroll
                    for (int i = 0; i < MT; ++i) {
                        if constexpr (ROWA)
                            break;  // k-contiguous rows: one 16-byte read below
                        const int m = mw + i * 32 + 16 * (g & 1) + 4 * (sl & 3);
                        ra[h][i] = trd(&Ad[buf][k * TM + (((m >> 3) ^ g1_swz16(k)) << 3) + (m & 7)]);
                    }
#pragma unroll
                    for (int j = 0; j < NT; ++j) {
                        const int n = nw + j * 32 + 16 * (g & 1) + 4 * (sl & 3);
                        rb[h][j] = trd(&Bd[buf][k * TN + (((n >> 3) ^ g1_swz16(k)) << 3) + (n & 7)]);
                    }
                }
#pragma unroll
                for (int i = 0; i < MT; ++i) {
                    if constexpr (ROWA) {
                        const int m = mw + i * 32 + (lane & 31);
                        av[kk][i] = *(const u16x8 *)&Ad[buf][m * TK + (((2 * kk + half) ^ g1_swzr(m)) << 3)];
                    } else {
                        av[kk][i] = __builtin_bit_cast(
                            u16x8, __builtin_shufflevector(ra[0][i], ra[1][i], 0, 1, 2, 3, 4, 5, 6, 7));
                    }
                }
#pragma unroll
                for (int j = 0; j < NT; ++j)
                    bv[kk][j] = __builtin_bit_cast(
                        u16x8, __builtin_shufflevector(rb[0][j], rb[1][j], 0, 1, 2, 3, 4, 5, 6, 7));
            }
            if (next)  // the next stage streams in during the MFMAs
                dload(k0 + TK, buf ^ 1);
#pragma unroll
            for (int kk = 0; kk < TK / 16; ++kk)
#pragma unroll
                for (int i = 0; i < MT; ++i)
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        acc[i][j] = mfma32x32x16bf(av[kk][i], bv[kk][j], acc[i][j]);
        } else if constexpr (DMA) {
            // operand k of MFMA c of 8-k block b8: 8 b8 + c (lanes 0-31) and
            // 8 b8 + 4 + c (lanes 32-63), as in the transposed layout
            float av[TK / 8][4][MT], bv[TK / 8][4][NT];
            if constexpr (ROWA) {  // k-contiguous rows: one 16-byte read per 8-k block
#pragma unroll
                for (int b8 = 0; b8 < TK / 8; ++b8)
#pragma unroll
                    for (int i = 0; i < MT; ++i) {
                        const int m = mw + i * 32 + (lane & 31);
                        const float4 v =
                            *(const float4 *)&Ad[buf][m * TK + (((2 * b8 + half) ^ g1_swzr(m)) << 2)];
                        av[b8][0][i] = v.x;
                        av[b8][1][i] = v.y;
                        av[b8][2][i] = v.z;
                        av[b8][3][i] = v.w;
                    }
            }
#pragma unroll
            for (int b8 = 0; b8 < TK / 8; ++b8)
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int k = 8 * b8 + 4 * half + c;
#pragma unroll
                    for (int i = 0; i < MT; ++i) {
                        if constexpr (ROWA)
                            break;
                        const int m = mw + i * 32 + (lane & 31);
                        av[b8][c][i] = Ad[buf][k * TM + ((((m >> 2) ^ g1_swz(k))) << 2) + (m & 3)];
                    }
#pragma unroll
                    for (int j = 0; j < NT; ++j) {
                        const int n = nw + j * 32 + (lane & 31);
                        bv[b8][c][j] = Bd[buf][k * TN + ((((n >> 2) ^ g1_swz(k))) << 2) + (n & 3)];
                    }
                }
            if (next)  // the next stage streams in during the MFMAs
                dload(k0 + TK, buf ^ 1);
#pragma unroll
            for (int b8 = 0; b8 < TK / 8; ++b8)
#pragma unroll
                for (int c = 0; c < 4; ++c)
#pragma unroll
                    for (int i = 0; i < MT; ++i)
#pragma unroll
                        for (int j = 0; j < NT; ++j)
                            acc[i][j] = mfma32x32x2(av[b8][c][i], bv[b8][c][j], acc[i][j]);
        } else if constexpr (!BF) {
            float4 av[TK / 8][MT], bv[TK / 8][NT];
#pragma unroll
            for (int b8 = 0; b8 < TK / 8; ++b8) {
#pragma unroll
                for (int i = 0; i < MT; ++i)
                    av[b8][i] = *(const float4 *)&As[buf][mw + i * 32 + (lane & 31)][8 * b8 + 4 * half];
#pragma unroll
                for (int j = 0; j < NT; ++j)
                    bv[b8][j] = *(const float4 *)&Bs[buf][nw + j * 32 + (lane & 31)][8 * b8 + 4 * half];
            }
#pragma unroll
            for (int b8 = 0; b8 < TK / 8; ++b8)
#pragma unroll
                for (int c = 0; c < 4; ++c)
#pragma unroll
                    for (int i = 0; i < MT; ++i)
#pragma unroll
                        for (int j = 0; j < NT; ++j)
                            acc[i][j] = mfma32x32x2(av[b8][i][c], bv[b8][j][c], acc[i][j]);
        } else {
            u16x8 av[TK / 16][MT], bv[TK / 16][NT];
#pragma unroll
            for (int kk = 0; kk < TK / 16; ++kk) {
#pragma unroll
                for (int i = 0; i < MT; ++i)
                    av[kk][i] = *(const u16x8 *)&As[buf][mw + i * 32 + (lane & 31)][16 * kk + 8 * half];
#pragma unroll
                for (int j = 0; j < NT; ++j)
                    bv[kk][j] = *(const u16x8 *)&Bs[buf][nw + j * 32 + (lane & 31)][16 * kk + 8 * half];
            }
#pragma unroll
            for (int kk = 0; kk < TK / 16; ++kk)
#pragma unroll
                for (int i = 0; i < MT; ++i)
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        acc[i][j] = mfma32x32x16bf(av[kk][i], bv[kk][j], acc[i][j]);
        }
        if (DMA)  // the next stage's lines are in LDS before anyone reads them
            __builtin_amdgcn_s_waitcnt(0);
        else if (next)
            stash(buf ^ 1);
        __syncthreads();
        buf ^= 1;
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

// FN (dense layout, fine structure with 32-row slices and 32-column blocks,
// BC = 32): a row group is one slice and a batch chunk is one block, so the
// chunks of removed blocks skip their MFMAs (exact zeros, bit-identical).
//
// DMA (B a multiple of BC, BC * element size = 128 bytes): the batch chunks go
// from global memory straight into LDS (global_load_lds_dwordx4, lane j of an
// instruction fills bytes [16 j, 16 j + 16) of a 1 KB block = 8 rows), with no
// register staging.  Rows are unpadded 128-byte lines whose 16-byte pieces are
// permuted per row (piece c of row r sits at c ^ wg_swz(r)) so that the
// operand reads of 16 consecutive rows hit distinct banks; the permutation is
// applied on the global side (each lane loads the piece its LDS slot holds).
// Rows past the end of the operands are clamped to a valid row: they only feed
// output rows or columns that are never stored.
__device__ __forceinline__ int wg_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }


// Sparse fp32 with DMA chunks and one 32-row temporary tile: operands staged
// half a chunk at a time; with at most two accumulator tiles three wavefronts
// per SIMD (register-bound otherwise at two; measured 4 % faster at H = 2048
// despite 36 bytes of spilled registers per lane), with four (75 % sparsity)
// two, which the half-chunk staging keeps from spilling.
template <typename TS, bool SPARSE, bool DMA, int TT, int ATN>
constexpr bool wg_splitop() { return SPARSE && DMA && sizeof(TS) == 4 && TT == 1; }
template <typename TS, bool SPARSE, bool DMA, int TT, int ATN>
constexpr int wg_occupancy() { return wg_splitop<TS, SPARSE, DMA, TT, ATN>() && ATN <= 2 ? 3 : 2; }

template <typename TS, bool SPARSE, int TT, int ATN, bool VEC, int BC, bool FN = false,
          bool DMA = false>
__global__ __launch_bounds__(THREADS, (wg_occupancy<TS, SPARSE, DMA, TT, ATN>())) void wgrad_kernel(WgradArgs a) {
    constexpr bool SPLITOP = wg_splitop<TS, SPARSE, DMA, TT, ATN>();
    static_assert(!(FN && (SPARSE || BC != 32 || TT != 1)), "fine chunks are 32-column blocks");
    static_assert(!DMA || (BC * sizeof(TS) == 128 && VEC), "DMA chunks are 128-byte lines");
    using E = typename std::conditional<sizeof(TS) == 4, float, uint16_t>::type;
    constexpr int PITCH = DMA ? BC : BC + (sizeof(TS) == 4 ? 4 : 8);
    constexpr int PE = 16 / sizeof(E);            // elements per 16-byte piece
    constexpr int GROWS = TT * 32;                // temporary-tile rows per group
    using V = Vec<TS, VEC>;
    constexpr int VW = V::W;
    constexpr int cpr = BC / VW;
    constexpr int gvec = WG_NG * GROWS * cpr, xvec = WG_FEAT * cpr;
    constexpr int RG = (gvec + THREADS - 1) / THREADS;
    constexpr int RX = (xvec + THREADS - 1) / THREADS;
    // two stages: the MFMAs read one while the next batch chunk is written to
    // the other (one barrier per chunk); the kept-slice table is kept per
    // step parity so that a step's routing never races the next step's table
    __shared__ __align__(16) E sX[2][WG_FEAT][PITCH];
    __shared__ __align__(16) E sG[2][WG_NG * GROWS][PITCH];
    __shared__ int sidx[2][WG_NG][64];

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
        int t0, t1, t2;
        geom(blockIdx.x * WG_NG + k, t0, t1, lc0[k], lcc[k], lq0[k], lqc[k], t2);
    }

    const int nbc = (B + BC - 1) / BC;
    const int niters = (a.t_end - a.t_begin) * nbc;

    // global -> register staging of one batch chunk; a vector never crosses
    // the end of a row (B is a multiple of VW when VEC).  Each thread's rows
    // are fixed for the whole launch, so their offsets within a step are
    // computed once; a chunk adds the step's base and the batch offset.
    // DMA: instruction k of a chunk fills rows [8k, 8k + 8) of sX (k < 16) or
    // of sG (k >= 16); wavefront w issues k = w, w + 4, ...
    constexpr int NDI = (WG_FEAT + WG_NG * GROWS) / 8, NDW = NDI / 4;
    static_assert(!DMA || (NDI % 4 == 0 && WG_FEAT == 128), "DMA instruction split");
    int dofs[DMA ? NDW : 1];
    bool disx[DMA ? NDW : 1];
    if constexpr (DMA) {
#pragma unroll
        for (int i = 0; i < NDW; ++i) {
            const int k = wave + 4 * i;
            const int rr = 8 * (k < 16 ? k : k - 16) + (lane >> 3);
            const int pc = (lane & 7) ^ wg_swz(rr);  // the piece this lane's LDS slot holds
            if (k < 16) {
                const int n = min(n0 + rr, NC - 1);
                disx[i] = n < I;
                dofs[i] = (n < I ? n : n - I) * B + pc * PE;
            } else {
                const int kk = rr / GROWS, lr = rr - kk * GROWS;
                const int crow = max(0, min(lc0[kk] + min(lr, max(lcc[kk] - 1, 0)), (int)a.Kp - 1));
                disx[i] = false;
                dofs[i] = crow * B + pc * PE;
            }
        }
    }
    V rg[DMA ? 1 : 2][DMA ? 1 : RG], rx[DMA ? 1 : 2][DMA ? 1 : RX];  // two chunks in flight
    int gofs[RG], gbb[RG], xofs[RX], xbb[RX];
    bool gok[RG], xok[RX], xisx[RX];
#pragma unroll
    for (int i = 0; i < RG; ++i) {
        const int q = tid + i * THREADS;
        const int rho = q / cpr, bb = (q - rho * cpr) * VW;
        const int k = rho / GROWS, lr = rho - k * GROWS;
        gok[i] = q < gvec && lr < lcc[k & (WG_NG - 1)];
        gofs[i] = (lc0[k & (WG_NG - 1)] + (gok[i] ? lr : 0)) * B + bb;
        gbb[i] = bb;
    }
#pragma unroll
    for (int i = 0; i < RX; ++i) {
        const int q = tid + i * THREADS;
        const int f = q / cpr, bb = (q - f * cpr) * VW;
        const int n = n0 + f;
        xok[i] = q < xvec && n < NC;
        xisx[i] = n < I;
        xofs[i] = (xisx[i] ? n : (xok[i] ? n - I : 0)) * B + bb;
        xbb[i] = bb;
    }
    int ridx[2] = {-1, -1};
    // steps run from t_end - 1 down to t_begin, and the launches of one call
    // go down in time too, so every row of dW sums its steps in one order
    // however the steps are split over launches
    auto load = [&](int it, int set, int lbuf) {
        const int tl = it / nbc, b0 = (it - tl * nbc) * BC;
        const int t = a.t_end - 1 - tl;
        const TS *Gt = Gc + (long)t * a.Kp * B + b0;
        const TS *xt = x + (long)t * I * B + b0;
        const TS *ht = h + (long)t * H * B + b0;
        if constexpr (DMA) {
#pragma unroll
            for (int i = 0; i < NDW; ++i) {
                const int k = wave + 4 * i;
                const TS *src = k < 16 ? (disx[i] ? xt : ht) + dofs[i] : Gt + dofs[i];
                E *dst = k < 16 ? &sX[lbuf][8 * k][0] : &sG[lbuf][8 * (k - 16)][0];
                __builtin_amdgcn_global_load_lds((glob_void_t *)src, (lds_void_t *)dst, 16, 0, 0);
            }
        } else {
#pragma unroll
            for (int i = 0; i < RG; ++i) {
                if (gok[i] && b0 + gbb[i] < B)
                    rg[DMA ? 0 : set][i].load(Gt + gofs[i], VW);
                else
                    rg[DMA ? 0 : set][i].zero();
            }
#pragma unroll
            for (int i = 0; i < RX; ++i) {
                if (xok[i] && b0 + xbb[i] < B)
                    rx[DMA ? 0 : set][i].load((xisx[i] ? xt : ht) + xofs[i], VW);
                else
                    rx[DMA ? 0 : set][i].zero();
            }
        }
        if (SPARSE && b0 == 0 && tid < WG_NG * 64) {
            const int k = tid >> 6, e = tid & 63;
            ridx[set] = e < lqc[k] ? a.idx[(long)t * a.kept + lq0[k] + e] : -1;
        }
        if (FN && b0 == 0 && tid < WG_NG * 64) {  // kept blocks of the group's slice
            const int k = tid >> 6, e = tid & 63;
            const long sl = (long)blockIdx.x * WG_NG + k;
            ridx[set] = (e < a.fkept && sl < G4 / 32)
                            ? a.fidx[((long)t * (G4 / 32) + sl) * a.fkept + e] : -1;
        }
    };
    auto stash = [&](int it, int set, int buf) {
        const int tl = it / nbc;
        if constexpr (!DMA) {
#pragma unroll
            for (int i = 0; i < RG; ++i) {
                const int q = tid + i * THREADS;
                if (q < gvec) {
                    const int rho = q / cpr, bb = (q - rho * cpr) * VW;
                    lds_store_vec(&sG[buf][rho][bb], rg[set][i]);
                }
            }
#pragma unroll
            for (int i = 0; i < RX; ++i) {
                const int q = tid + i * THREADS;
                if (q < xvec) {
                    const int f = q / cpr, bb = (q - f * cpr) * VW;
                    lds_store_vec(&sX[buf][f][bb], rx[set][i]);
                }
            }
        }
        if ((SPARSE || FN) && it - tl * nbc == 0 && tid < WG_NG * 64)
            sidx[tl & 1][tid >> 6][tid & 63] = ridx[set];
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
    // a later launch of the same call continues the sums of the earlier ones
    // from the stored dW (the same fp32 additions as one launch)
    if (a.accumulate) {
#pragma unroll
        for (int at = 0; at < ATN; ++at) {
            if (at >= AT)
                break;
            const int col = at * 32 + (lane & 31);
            if (col >= rcount)
                continue;
            const float *src = a.dW + (long)(r0 + col) * NC;
#pragma unroll
            for (int ft = 0; ft < WG_FT; ++ft)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int f = n0 + fh * 64 + ft * 32 + acc_row(lane, v);
                    if (f < NC)
                        acc[ft][at][v] = src[f];
                }
        }
    }

    load(0, 0, 0);
    if (!DMA && niters > 1)
        load(1, 1, 1);
    stash(0, 0, 0);
    if (DMA)
        __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    constexpr int HALF = BC / 2;
    const int hb = (lane >> 5) * HALF;
    // iteration it computes from LDS buffer it & 1, loads chunk it + 2 into
    // register set it & 1 and stores chunk it + 1 (set and buffer
    // (it + 1) & 1); the loop runs in pairs so that the sets are static
    uint64_t fmask = ~0ull;  // FN: kept blocks of this wavefront's slice at the current step

    // sparse routing: csrc[at] is the temporary column (kept row) that
    // accumulator column at * 32 + lane pulls at the current step, -1 if its
    // slice was dropped.  (Routing a step during the next step's first chunk,
    // to overlap the permutes with MFMAs, measured no faster.)
    int csrc[ATN];
    auto lookup = [&](int tl) {
        const int *tab = sidx[tl & 1][gi];
#pragma unroll
        for (int at = 0; at < ATN; ++at) {
            const int col = at * 32 + (lane & 31);
            int src = -1;
            if (col < rcount) {
                const int orow = r0 + col;
                const int js = orow / a.P;
                const int reg = (js - j0) / a.R;
                const int e0 = reg * ks, e1 = min(e0 + ks, qcount);
                for (int e = e0; e < e1; ++e)
                    if (tab[e] == js)
                        src = e * a.P + (orow - js * a.P);
            }
            csrc[at] = src;
        }
    };
    // acc[:, at] += t routed by srcs (accumulator tiles past the group's rows
    // have src -1 everywhere and stay zero)
    auto route = [&](const f32x16 (&t)[WG_FT][TT], const int (&srcs)[ATN]) {
#pragma unroll
        for (int at = 0; at < ATN; ++at) {
            const int src = srcs[at];
            const int saddr = (((src < 0 ? 0 : src) & 31) + (lane & 32)) << 2;
            const int stile = src < 0 ? 0 : (src >> 5);
#pragma unroll
            for (int ft = 0; ft < WG_FT; ++ft) {
                // all lane permutes of this feature tile first, then the adds
                float val[TT][16];
#pragma unroll
                for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        val[tt][v] = __int_as_float(
                            __builtin_amdgcn_ds_bpermute(saddr, __float_as_int(t[ft][tt][v])));
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    float w = val[0][v];
                    if (TT > 1)
                        w = stile == 1 ? val[TT > 1 ? 1 : 0][v] : w;
                    acc[ft][at][v] += src < 0 ? 0.f : w;  // dropped: exactly 0, even for inf/NaN
                }
            }
        }
    };

    auto iter = [&](int it, auto sc) {
        constexpr int S0 = decltype(sc)::value, S1 = 1 - S0;
        const int buf = S0;
        const int tl = it / nbc, bc = it - tl * nbc;
        if (!DMA && it + 2 < niters)
            load(it + 2, S0, 0);
        // DMA: the next chunk streams into the other buffer (read in the
        // previous iteration), issued once this chunk's operands are in
        // registers (a deeper, three-buffer pipeline measured slower)
        auto issue_next = [&]() {
            if (DMA && it + 1 < niters)
                load(it + 1, S1, S1);
        };
        if constexpr (FN) {
            if (bc == 0) {
                const int v = sidx[tl & 1][gi][lane];
                uint64_t m = v >= 0 ? (1ull << v) : 0ull;
#pragma unroll
                for (int off = 32; off >= 1; off >>= 1) {
                    const uint32_t lo = __shfl_xor((uint32_t)m, off, 64);
                    const uint32_t hi = __shfl_xor((uint32_t)(m >> 32), off, 64);
                    m |= ((uint64_t)hi << 32) | lo;
                }
                fmask = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(m >> 32)) << 32) |
                        __builtin_amdgcn_readfirstlane((uint32_t)m);
            }
        }
        const bool run = !FN || !a.fskip || ((fmask >> bc) & 1);
        // column (element) of the 16-byte piece p of LDS row r
        auto pcol = [&](int r, int p) { return DMA ? (p ^ wg_swz(r)) * PE : p * PE; };

        // MFMA over this batch chunk: WG_FT feature tiles x TT row tiles
        if (!run) {
            // removed block: its products are zero
            issue_next();
        } else if constexpr (sizeof(TS) == 4 && SPLITOP) {
            // operands of half the chunk at a time (fewer live registers)
            issue_next();  // the next chunks stream in during the MFMAs
#pragma unroll
            for (int sh = 0; sh < HALF / 4; sh += 2) {
                float4 av[2][WG_FT], bv[2][TT];
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2) {
#pragma unroll
                    for (int ft = 0; ft < WG_FT; ++ft) {
                        const int r = fh * 64 + ft * 32 + (lane & 31);
                        av[s2][ft] = *(const float4 *)&sX[buf][r][pcol(r, hb / 4 + sh + s2)];
                    }
#pragma unroll
                    for (int tt = 0; tt < TT; ++tt) {
                        const int r = gi * GROWS + tt * 32 + (lane & 31);
                        bv[s2][tt] = *(const float4 *)&sG[buf][r][pcol(r, hb / 4 + sh + s2)];
                    }
                }
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
                    for (int c4 = 0; c4 < 4; ++c4)
#pragma unroll
                        for (int ft = 0; ft < WG_FT; ++ft)
#pragma unroll
                            for (int tt = 0; tt < TT; ++tt)
                                tmp[ft][tt] = mfma32x32x2(av[s2][ft][c4], bv[s2][tt][c4], tmp[ft][tt]);
            }
        } else if constexpr (sizeof(TS) == 4) {
            float4 av[HALF / 4][WG_FT], bv[HALF / 4][TT];
#pragma unroll
            for (int s = 0; s < HALF / 4; ++s) {
#pragma unroll
                for (int ft = 0; ft < WG_FT; ++ft) {
                    const int r = fh * 64 + ft * 32 + (lane & 31);
                    av[s][ft] = *(const float4 *)&sX[buf][r][pcol(r, hb / 4 + s)];
                }
#pragma unroll
                for (int tt = 0; tt < TT; ++tt) {
                    const int r = gi * GROWS + tt * 32 + (lane & 31);
                    bv[s][tt] = *(const float4 *)&sG[buf][r][pcol(r, hb / 4 + s)];
                }
            }
            issue_next();  // the next chunks stream in during the MFMAs
#pragma unroll
            for (int s = 0; s < HALF / 4; ++s)
#pragma unroll
                for (int c4 = 0; c4 < 4; ++c4)
#pragma unroll
                    for (int ft = 0; ft < WG_FT; ++ft)
#pragma unroll
                        for (int tt = 0; tt < TT; ++tt)
                            tmp[ft][tt] = mfma32x32x2(av[s][ft][c4], bv[s][tt][c4], tmp[ft][tt]);
        } else {
            u16x8 av[HALF / 8][WG_FT], bv[HALF / 8][TT];
#pragma unroll
            for (int s = 0; s < HALF / 8; ++s) {
#pragma unroll
                for (int ft = 0; ft < WG_FT; ++ft) {
                    const int r = fh * 64 + ft * 32 + (lane & 31);
                    av[s][ft] = *(const u16x8 *)&sX[buf][r][pcol(r, hb / 8 + s)];
                }
#pragma unroll
                for (int tt = 0; tt < TT; ++tt) {
                    const int r = gi * GROWS + tt * 32 + (lane & 31);
                    bv[s][tt] = *(const u16x8 *)&sG[buf][r][pcol(r, hb / 8 + s)];
                }
            }
            issue_next();
#pragma unroll
            for (int s = 0; s < HALF / 8; ++s)
#pragma unroll
                for (int ft = 0; ft < WG_FT; ++ft)
#pragma unroll
                    for (int tt = 0; tt < TT; ++tt)
                        tmp[ft][tt] = mfma32x32x16bf(av[s][ft], bv[s][tt], tmp[ft][tt]);
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
                lookup(tl);
                route(tmp, csrc);
#pragma unroll
                for (int ft = 0; ft < WG_FT; ++ft)
#pragma unroll
                    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                        for (int v = 0; v < 16; ++v)
                            tmp[ft][tt][v] = 0.f;
            }
        }
        if (it + 1 < niters)
            stash(it + 1, S1, S1);
        if (DMA)  // the next chunk's lines are in LDS before anyone reads them
            __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    };
    int it0 = 0;
    for (; it0 + 1 < niters; it0 += 2) {
        iter(it0, std::integral_constant<int, 0>{});
        iter(it0 + 1, std::integral_constant<int, 1>{});
    }
    if (it0 < niters)
        iter(it0, std::integral_constant<int, 0>{});

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
                    dst[f] = acc[ft][at][v];
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

// Tile of the data-gradient GEMM.  Its operands stream from L2 / MALL, so
// occupancy matters as much as operand reuse: fp32 runs 128 x 128 tiles
// when those still give every CU a work-group (short-k split launches),
// else 64 x 64 (three work-groups per CU); bf16, whose MFMA is 8x faster per
// byte staged, always runs 128-row tiles.
void gemm1_tile(bool bf16, int N, long rows, long zdim, int *tm, int *tn) {
    if (N <= 32) {
        *tm = 128;
        *tn = 32;
    } else if (N <= 64) {
        *tm = bf16 ? 128 : 64;
        *tn = 64;
    } else if (bf16 || ceil_div(rows, 128) * ceil_div(N, 128) * zdim >= 256) {
        *tm = 128;
        *tn = 128;
    } else {
        *tm = 64;
        *tn = 64;
    }
}

// Work-groups of one data-gradient tile configuration resident per CU
// (bounded by its LDS: two stages of (TM + TN) rows of 144 bytes plus the
// gathered-row table, out of 160 KiB).
int gemm1_wgs_per_cu(int tm, int tn) {
    const long lds = 2L * (tm + tn) * 144 + 4L * GEMM1_KC_MAX;
    return (int)std::max(1L, (160L * 1024) / lds);
}

template <typename TS, int TM, int TN, bool GA, bool VE, bool ROWA = false>
static void launch_g1(dim3 grid, const Gemm1Args &a, bool w8, hipStream_t s, bool dma = false) {
    if constexpr (sizeof(TS) == 4 && VE && TN != 32) {
        if (dma && !w8) {
            hipLaunchKernelGGL((gemm1_kernel<TS, TM, TN, GA, true, ROWA, 4, false, true>), grid,
                               dim3(THREADS), 0, s, a);
            return;
        }
    }
    if constexpr (sizeof(TS) == 2 && VE && TM == 128 && TN == 128) {
        if (dma && w8) {
            hipLaunchKernelGGL((gemm1_kernel<TS, 128, 128, GA, true, ROWA, 8, false, true>), grid,
                               dim3(512), 0, s, a);
            return;
        }
    }
    if constexpr (!GA && !ROWA && TM == 128 && TN == 32) {
        if (a.fidx) {
            hipLaunchKernelGGL((gemm1_kernel<TS, 128, 32, false, VE, false, 4, true>), grid, dim3(THREADS), 0, s, a);
            return;
        }
    }
    if constexpr (TM == 128 && TN == 128) {
        if (w8) {
            hipLaunchKernelGGL((gemm1_kernel<TS, TM, TN, GA, VE, ROWA, 8>), grid, dim3(512), 0, s, a);
            return;
        }
    }
    hipLaunchKernelGGL((gemm1_kernel<TS, TM, TN, GA, VE, ROWA>), grid, dim3(THREADS), 0, s, a);
}

// Wavefronts per work-group: 128 x 128 bf16 tiles run eight (two per SIMD
// per work-group; bf16 MFMAs finish 8x faster per staged byte than fp32, so
// they need more wavefronts to cover load latency: measured 1.35-1.5x on the
// H = 4096, B = 256 products), everything else four, unless a.waves says.
static bool use_w8(const Gemm1Args &a, bool bf16, int TM, int TN) {
    if (TM != 128 || TN != 128)
        return false;
    return a.waves == 8 || (a.waves == 0 && bf16);
}

hipError_t launch_gemm1(Gemm1Args a, bool bf16, hipStream_t s) {
    if (a.k_chunk % GEMM1_TK != 0 || a.splitk < 1 || a.steps < 1)
        return hipErrorInvalidValue;
    // fine fast path: no gather, whole 32-row slices, 32-column blocks, the
    // slice masks of one split fit the work-group's table
    if (a.fidx && (a.idx || a.P != 32 || a.fkept < 1 || a.fkept > 64 || a.N % 32 != 0 ||
                   ceil_div(a.k_chunk, 32) > FINE_MAX_SLICES))
        return hipErrorInvalidValue;
    // 16-byte vector loads need 16-byte aligned rows; the tile origin is
    // rounded down to the vector width and rows below m_begin are not stored
    const int vw = bf16 ? 8 : 4;
    const bool vec = a.ldw % vw == 0 && a.N % vw == 0;
    a.m_lo = vec ? a.m_begin / vw * vw : a.m_begin;
    const long z = (long)a.splitk * a.steps;
    // DMA stages: whole k stages (32 fp32 or 64 bf16 rows), 16-byte aligned rows
    const bool dma_shape = a.dma && vec && !a.fidx && a.Kp % (bf16 ? 64 : 32) == 0 &&
                           ((uintptr_t)a.W & 15) == 0 && ((uintptr_t)a.Gc & 15) == 0;
    int TM, TN;
    gemm1_tile(bf16, a.N, a.M - a.m_lo, z, &TM, &TN);
    if (dma_shape && !bf16 && a.N > 32) {  // fp32 DMA stages: the 64 x 64 tile measured best throughout
        TM = 64;
        TN = 64;
    }
    if (a.tm)
        TM = a.tm;
    if (a.tn)
        TN = a.tn;
    if (a.fidx) {  // one column block per work-group
        TM = 128;
        TN = 32;
    }
    if (!((TN == 32 && TM == 128) || ((TN == 64 || TN == 128) && (TM == 64 || TM == 128))))
        return hipErrorInvalidValue;
    dim3 grid((unsigned)ceil_div(a.M - a.m_lo, TM), (unsigned)ceil_div(a.N, TN), (unsigned)z);
    const bool gather = a.idx != nullptr;
    if (a.waves != 0 && a.waves != 4 && !(a.waves == 8 && TM == 128 && TN == 128))
        return hipErrorInvalidValue;
    const bool w8 = use_w8(a, bf16, TM, TN);
    const bool dma = dma_shape && (bf16 ? (w8 && TM == 128 && TN == 128) : TN != 32);
#define LSTMSS_G1(TS, TMV, TNV, GA, VE) launch_g1<TS, TMV, TNV, GA, VE>(grid, a, w8, s, dma)
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

hipError_t launch_gemm_fwd(Gemm1Args a, bool bf16, hipStream_t s) {
    if (a.k_chunk % GEMM1_TK != 0 || a.splitk < 1 || a.steps < 1 || a.idx || a.m_begin != 0)
        return hipErrorInvalidValue;
    const int vw = bf16 ? 8 : 4;
    const bool vec = a.ldw % vw == 0 && a.kcol0 % vw == 0 && a.N % vw == 0;
    a.m_lo = 0;
    const long z = (long)a.splitk * a.steps;
    // DMA stages: whole k stages of the product (K' = a.Kp rows), 16-byte aligned rows
    const bool dma_shape = a.dma && vec && a.Kp % (bf16 ? 64 : 32) == 0 &&
                           a.k_chunk % (bf16 ? 64 : 32) == 0 && ((uintptr_t)a.W & 15) == 0 &&
                           ((uintptr_t)a.Gc & 15) == 0;
    int TM, TN;
    gemm1_tile(bf16, a.N, a.M, z, &TM, &TN);
    if (dma_shape && !bf16 && a.N > 32) {  // fp32 DMA stages: 64 x 64 tiles, as in launch_gemm1
        TM = 64;
        TN = 64;
    }
    if (a.tm)
        TM = a.tm;
    if (a.tn)
        TN = a.tn;
    if (!((TN == 32 && TM == 128) || ((TN == 64 || TN == 128) && (TM == 64 || TM == 128))))
        return hipErrorInvalidValue;
    dim3 grid((unsigned)ceil_div(a.M, TM), (unsigned)ceil_div(a.N, TN), (unsigned)z);
    if (a.waves != 0 && a.waves != 4 && !(a.waves == 8 && TM == 128 && TN == 128))
        return hipErrorInvalidValue;
    const bool w8 = use_w8(a, bf16, TM, TN);
    const bool dma = dma_shape && (bf16 ? (w8 && TM == 128 && TN == 128) : TN != 32);
#define LSTMSS_GF(TS, TMV, TNV, VE) launch_g1<TS, TMV, TNV, false, VE, true>(grid, a, w8, s, dma)
#define LSTMSS_GFV(TS, TMV, TNV) do { if (vec) LSTMSS_GF(TS, TMV, TNV, true); else LSTMSS_GF(TS, TMV, TNV, false); } while (0)
#define LSTMSS_GFT(TS) do { \
        if (TN == 32) LSTMSS_GFV(TS, 128, 32); \
        else if (TN == 64) { if (TM == 128) LSTMSS_GFV(TS, 128, 64); else LSTMSS_GFV(TS, 64, 64); } \
        else { if (TM == 128) LSTMSS_GFV(TS, 128, 128); else LSTMSS_GFV(TS, 64, 128); } } while (0)
    if (bf16) LSTMSS_GFT(bf16_t); else LSTMSS_GFT(float);
#undef LSTMSS_GFT
#undef LSTMSS_GFV
#undef LSTMSS_GF
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

// One weight-gradient launch; `dma` takes the LDS-DMA variant (128-byte
// chunks: 32 fp32 or 64 bf16 batch columns).
template <typename TS, bool SP, int TTV, int ATV, bool FN>
static void wg_launch(const WgradArgs &a, bool vec, bool dma, dim3 grid, hipStream_t s) {
    constexpr int DBC = 128 / (int)sizeof(TS);
    if constexpr (!FN || DBC == 32) {
        if (dma) {
            hipLaunchKernelGGL((wgrad_kernel<TS, SP, TTV, ATV, true, DBC, FN, true>), grid,
                               dim3(THREADS), 0, s, a);
            return;
        }
    }
    if constexpr (FN) {
        if (vec)
            hipLaunchKernelGGL((wgrad_kernel<TS, false, 1, 1, true, 32, true>), grid, dim3(THREADS), 0, s, a);
        else
            hipLaunchKernelGGL((wgrad_kernel<TS, false, 1, 1, false, 32, true>), grid, dim3(THREADS), 0, s, a);
    } else {
#define LSTMSS_WG(VE) do { \
        if (a.BC == 16) hipLaunchKernelGGL((wgrad_kernel<TS, SP, TTV, ATV, VE, 16>), grid, dim3(THREADS), 0, s, a); \
        else if (a.BC == 32) hipLaunchKernelGGL((wgrad_kernel<TS, SP, TTV, ATV, VE, 32>), grid, dim3(THREADS), 0, s, a); \
        else hipLaunchKernelGGL((wgrad_kernel<TS, SP, TTV, ATV, VE, 64>), grid, dim3(THREADS), 0, s, a); } while (0)
        if (vec)
            LSTMSS_WG(true);
        else
            LSTMSS_WG(false);
#undef LSTMSS_WG
    }
}

static bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }

hipError_t launch_wgrad(WgradArgs a, bool sparse, bool bf16, hipStream_t s) {
    const int es = bf16 ? 2 : 4;
    // the LDS-DMA variant: whole 128-byte chunks of 16-byte aligned rows
    auto dma_ok = [&](int bc) {
        return a.dma && bc * es == 128 && a.B % bc == 0 && aligned16(a.Gc) && aligned16(a.x) &&
               aligned16(a.h);
    };
    if (a.fidx) {  // fine structure, 32-row slices x 32-column blocks
        if (sparse || a.B % 32 != 0 || a.fkept < 1 || a.fkept > 64 || (4L * a.H) % 32 != 0)
            return hipErrorInvalidValue;
        a.BC = 32;
        const bool vec = a.B % (bf16 ? 8 : 4) == 0;
        dim3 grid((unsigned)ceil_div(ceil_div(4L * a.H, 32), WG_NG),
                  (unsigned)ceil_div(a.I + a.H, WG_FEAT));
        if (bf16)
            wg_launch<bf16_t, false, 1, 1, true>(a, vec, false, grid, s);
        else
            wg_launch<float, false, 1, 1, true>(a, vec, dma_ok(32), grid, s);
        return hipGetLastError();
    }
    int tt = 1, at = 1;
    if (sparse) {
        if (!wgrad_supported(a.P, a.R, a.S))
            return hipErrorNotSupported;
        wgrad_tiles(a.P, a.R, a.S, &a.greg, &tt, &at);
    }
    // batch columns per stage: 16/32 (fp32) or 32/64 (bf16, whole MFMA
    // k-blocks); larger stages would not leave room for two wavefronts per SIMD
    const int bc = a.B <= 16 ? 16 : a.B <= 32 ? 32 : (bf16 ? 64 : 32);
    a.BC = bc;
    const int vw = bf16 ? 8 : 4;
    const bool vec = a.B % vw == 0;
    const bool dma = dma_ok(bc);
    const long groups = sparse ? ceil_div(ceil_div(4L * a.H / a.P, a.R), a.greg) : ceil_div(4L * a.H, 32);
    dim3 grid((unsigned)ceil_div(groups, WG_NG), (unsigned)ceil_div(a.I + a.H, WG_FEAT));
#define LSTMSS_WGA(TS, TTV) do { \
        if (at <= 1) wg_launch<TS, true, TTV, 1, false>(a, vec, dma, grid, s); \
        else if (at <= 2) wg_launch<TS, true, TTV, 2, false>(a, vec, dma, grid, s); \
        else wg_launch<TS, true, TTV, 4, false>(a, vec, dma, grid, s); } while (0)
    if (bf16) {
        if (!sparse) wg_launch<bf16_t, false, 1, 1, false>(a, vec, dma, grid, s);
        else if (tt == 1) LSTMSS_WGA(bf16_t, 1);
        else LSTMSS_WGA(bf16_t, 2);
    } else {
        if (!sparse) wg_launch<float, false, 1, 1, false>(a, vec, dma, grid, s);
        else if (tt == 1) LSTMSS_WGA(float, 1);
        else LSTMSS_WGA(float, 2);
    }
#undef LSTMSS_WGA
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
