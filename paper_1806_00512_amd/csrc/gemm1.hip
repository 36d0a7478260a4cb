// Data-gradient MFMA product on the compacted gate gradient, and the forward
// products (input projection of all steps, split recurrent product).
//
// Paper: the gate gradient feeds every weight and data gradient product of
// the LSTM backward pass (section 3); after sparsifying, the kept slices are
// a dense matrix plus an offset index array, so the products run as dense
// block GEMMs that read the kept rows of W through the index (section 3 after
// Fig. 2, section 4).  Here:
//   data gradient    [dx_t; dh_{t-1}] = W_c^T dG_c   (W_c = kept rows of W)
//
// Tiles are 64-wide-wavefront MFMA tiles (32x32 outputs per wave), staged
// through LDS.  fp32 uses v_mfma_f32_32x32x2f32; bf16 uses
// v_mfma_f32_32x32x16_bf16 with fp32 accumulation.
#include "gemm_common.h"
#include "select.h"

namespace lstmss {

namespace {

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

// SEL: the coarse selection of one step inside its dh product.  Every
// work-group ranks the slices of its split's regions (whole regions: the
// split length is a multiple of P (R - S) kept rows) from the element
// kernel's chunk sums of squares, with the same wavefront routines as the
// select kernel, and gathers the rows of both operands through the result:
// W rows and the staging matrix's rows (Gc).  The split's work-groups share
// out the copy of its kept rows to the compacted matrix (after their
// product, from the staging matrix); those of tile (0, 0) also write the
// split's slots of the offset index.
template <typename TS, int TM, int TN, bool GATHER, bool VEC, bool ROWA = false, int NW = 4,
          bool FN = false, bool DMA = false, bool SEL = false>
__global__ __launch_bounds__(NW * 64) void gemm1_kernel(Gemm1Args a) {
    static_assert(!(ROWA && GATHER), "the forward products read every row");
    static_assert(!SEL || (DMA && GATHER), "selection in the product: gathered DMA stages");
    static_assert(!(FN && (GATHER || ROWA)), "the fine fast path reads every row");
    static_assert(!DMA || (VEC && (!FN || (sizeof(TS) == 4 && TM == 128 && TN == 32)) &&
                           (sizeof(TS) == 4 ? NW == 4 : (NW == 8 && TM == 128 && TN == 128))),
                  "DMA stages: fp32 products (the fine path with 128 x 32 tiles), or bf16 "
                  "128 x 128 tiles of eight wavefronts");
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
            srow[i] = GATHER ? idx[k / a.P] * a.P + k % a.P : (FN ? grow(k) : k);
        }
    };
    __shared__ __align__(16) E As[2][DMA ? 1 : TM][LDK];
    __shared__ __align__(16) E Bs[2][DMA ? 1 : TN][LDK];
    __shared__ __align__(16) E Ad[2][DMA ? TK * TM : 1];  // DMA: [k][m]
    __shared__ __align__(16) E Bd[2][DMA ? TK * TN : 1];  // DMA: [k][n]
    if constexpr (SEL) {
        const int P = a.P, R = a.sel_R, S = a.sel_S, kr = P * (R - S), nch = a.sel_nch;
        const long s_lo = (long)(kb / kr) * R;
        const long s_hi = ke0 == a.Kp ? a.sel_nslices : min(a.sel_nslices, (long)(ke0 / kr) * R);
        const int gs = (64 / R) * R;  // whole regions per wavefront
        const int ng = (int)((s_hi - s_lo + gs - 1) / gs);
        const bool write_idx = blockIdx.x == 0 && blockIdx.y == 0;
        // A group's chunk sums (L per slice) are one contiguous run: a
        // wavefront reads it coalesced into its own region of the stage
        // buffers (free until the first stage), lane j's slice at row j,
        // its entries permuted by j when L is a power of two so that the
        // lanes' reads of one entry fall on distinct banks; then each lane
        // folds its slice as select_slices does.  With fewer than 16 entries
        // per slice (measured faster so), or without room for a region, the
        // lanes read their slices directly.
        const int L = P * nch, rsb = 64 * L * (int)sizeof(double);
        const int na = (int)(sizeof(Ad) / rsb);
        const int nact = L < 16 ? 0 : min(NW, na + (int)(sizeof(Bd) / rsb));
        const bool pow2 = (L & (L - 1)) == 0;
        const int lg = __builtin_ctz(L);
        auto pos = [&](int j, int e) { return j * L + (pow2 ? e ^ (j & (L - 1)) : e); };
        const int gstep = nact > 0 ? nact : NW;
        for (int g = wave; wave < gstep && g < ng; g += gstep) {
            const long j0 = s_lo + (long)g * gs;
            const int nsl = (int)min((long)gs, s_hi - j0);
            SliceSel sl;
            if (nact > 0) {
                double *sq = (double *)(wave < na ? (char *)&Ad[0][0] + wave * rsb
                                                  : (char *)&Bd[0][0] + (wave - na) * rsb);
                const double *src = a.sel_sq + j0 * P * nch;
                const int n = nsl * L;
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the previous group's reads
                for (int x0 = 0; x0 < n; x0 += 8 * 64) {
                    double v[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        const int x = x0 + u * 64 + lane;
                        v[u] = x < n ? src[x] : 0.0;
                    }
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        const int x = x0 + u * 64 + lane;
                        const int j = pow2 ? x >> lg : x / L;
                        if (x < n)
                            sq[pos(j, x - j * L)] = v[u];
                    }
                }
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the wavefront's writes landed
                double scv = 0.0;
                if (lane < nsl) {
                    for (int p = 0; p < P; ++p) {
                        double rs = sq[pos(lane, p * nch)];
                        for (int c = 1; c < nch; ++c)
                            rs = rs + sq[pos(lane, p * nch + c)];
                        scv = p == 0 ? rs : scv + rs;
                    }
                }
                sl = rank_slices(scv, j0, nsl, R, S, a.sel_nslices);
            } else {
                sl = select_slices(a.sel_sq, nch, j0, nsl, P, R, S, a.sel_nslices);
            }
            if (sl.slot >= 0) {
                const int j = (int)(j0 + lane);
                for (int p = 0; p < P; ++p)
                    srow[sl.slot * P + p - kb] = j * P + p;
                if (write_idx)
                    a.sel_idx[sl.slot] = j;
            }
        }
    } else if (!ROWA && (!FN || DMA)) {  // FN with DMA stages: the kept slices' rows
        fill_rows(sc);
    }

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
            // 32-column rows (128 bytes) cannot be split: the second operand's
            // rows go to the slots of each group of 8 in the order k, k + 4,
            // k + 1, k + 5, ..., so that the rows k and k + 4 a wavefront reads
            // together are adjacent (distinct banks); the slot kl holds row kg
            const bool nsw = !isa && TN == 32;
            const int kg = nsw ? (kl & ~7) + ((kl & 7) >> 1) + 4 * (kl & 1) : kl;
            const int col = (nsw ? pc : pc ^ swz(kl)) * PEL;  // first column this lane's slot holds
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
                src = G + (long)((SEL || FN) ? srow[k0 + kg - sc] : k0 + kg) * N + n;
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
        if (ke > kb)  // FN: a block no slice of the range keeps has no stages
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
            if (!ROWA && (!FN || DMA) && !SEL && k0 + TK == sc + GEMM1_KC_MAX) {  // next super-chunk of rows
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
                        if constexpr (TN == 32)  // row k in slot (k & ~7) + 2 (k & 3) + ((k >> 2) & 1)
                            bv[b8][c][j] = Bd[buf][((k & ~7) + 2 * (k & 3) + ((k >> 2) & 1)) * TN + n];
                        else
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

    // SEL: compacted rows.  The split's rows are shared out over its
    // m-tiles, each work-group copying its share (its columns) from the
    // staging matrix after its product, so that no stage waits for these
    // stores; the first pieces are loaded before the partial sums are
    // stored, so that waiting for them does not wait for those stores.
    constexpr int PPR = TN / PEL;  // 16-byte pieces per tile row
    constexpr int CPB = SEL ? 2 : 1;
    uint4 cbuf[CPB];
    int c_r0 = 0, c_np = 0;
    if constexpr (SEL) {
        const int nr = ke0 - kb, nmt = (int)gridDim.x;
        c_r0 = (int)((long)nr * blockIdx.x / nmt);
        c_np = ((int)((long)nr * (blockIdx.x + 1) / nmt) - c_r0) * PPR;
#pragma unroll
        for (int i = 0; i < CPB; ++i) {
            const int e = tid + i * THREADS;
            const int k = kb + c_r0 + e / PPR, n = n0 + (e % PPR) * PEL;
            cbuf[i] = make_uint4(0, 0, 0, 0);
            if (e < c_np && n < N)
                cbuf[i] = *(const uint4 *)(G + (long)srow[k - sc] * N + n);
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
    if constexpr (SEL) {
        TS *gc = (TS *)a.sel_gc;
#pragma unroll
        for (int i = 0; i < CPB; ++i) {
            const int e = tid + i * THREADS;
            const int k = kb + c_r0 + e / PPR, n = n0 + (e % PPR) * PEL;
            if (e < c_np && n < N)
                *(uint4 *)(gc + (long)k * N + n) = cbuf[i];
        }
        for (int e = tid + CPB * THREADS; e < c_np; e += THREADS) {
            const int k = kb + c_r0 + e / PPR, n = n0 + (e % PPR) * PEL;
            if (n < N)
                *(uint4 *)(gc + (long)k * N + n) = *(const uint4 *)(G + (long)srow[k - sc] * N + n);
        }
    }
}

} // namespace

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
            if constexpr (GA && !ROWA) {
                if (a.sel_sq) {
                    hipLaunchKernelGGL((gemm1_kernel<TS, TM, TN, true, true, false, 4, false, true, true>),
                                       grid, dim3(THREADS), 0, s, a);
                    return;
                }
            }
            hipLaunchKernelGGL((gemm1_kernel<TS, TM, TN, GA, true, ROWA, 4, false, true>), grid,
                               dim3(THREADS), 0, s, a);
            return;
        }
    }
    if constexpr (sizeof(TS) == 2 && VE && TM == 128 && TN == 128) {
        if (dma && w8) {
            if constexpr (GA && !ROWA) {
                if (a.sel_sq) {
                    hipLaunchKernelGGL((gemm1_kernel<TS, 128, 128, true, true, false, 8, false, true, true>),
                                       grid, dim3(512), 0, s, a);
                    return;
                }
            }
            hipLaunchKernelGGL((gemm1_kernel<TS, 128, 128, GA, true, ROWA, 8, false, true>), grid,
                               dim3(512), 0, s, a);
            return;
        }
    }
    if constexpr (!GA && !ROWA && TM == 128 && TN == 32) {
        if (a.fidx) {
            if constexpr (sizeof(TS) == 4 && VE) {
                if (dma) {
                    hipLaunchKernelGGL((gemm1_kernel<TS, 128, 32, false, true, false, 4, true, true>), grid,
                                       dim3(THREADS), 0, s, a);
                    return;
                }
            }
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

// Launch configuration of a data-gradient product (sets a.m_lo).
struct G1Plan {
    int TM, TN;
    bool vec, w8, dma;
    dim3 grid;
};

static hipError_t g1_plan(Gemm1Args &a, bool bf16, G1Plan *pl) {
    if (a.k_chunk % GEMM1_TK != 0 || a.splitk < 1 || a.steps < 1)
        return hipErrorInvalidValue;
    // fine fast path: no gather, whole 32-row slices, 32-column blocks, the
    // slice masks of one split fit the work-group's table
    if (a.fidx && (a.idx || a.sel_sq || a.P != 32 || a.fkept < 1 || a.fkept > 64 ||
                   a.N % 32 != 0 || ceil_div(a.k_chunk, 32) > FINE_MAX_SLICES))
        return hipErrorInvalidValue;
    // 16-byte vector loads need 16-byte aligned rows; the tile origin is
    // rounded down to the vector width and rows below m_begin are not stored
    const int vw = bf16 ? 8 : 4;
    const bool vec = a.ldw % vw == 0 && a.N % vw == 0;
    a.m_lo = vec ? a.m_begin / vw * vw : a.m_begin;
    const long z = (long)a.splitk * a.steps;
    // DMA stages: whole k stages (32 fp32 or 64 bf16 rows), 16-byte aligned rows
    const bool dma_shape = a.dma && vec && (!a.fidx || !bf16) && a.Kp % (bf16 ? 64 : 32) == 0 &&
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
    if (a.waves != 0 && a.waves != 4 && !(a.waves == 8 && TM == 128 && TN == 128))
        return hipErrorInvalidValue;
    pl->TM = TM;
    pl->TN = TN;
    pl->vec = vec;
    pl->w8 = use_w8(a, bf16, TM, TN);
    // fp32 DMA stages: 64- and 128-column tiles, and the fine path's 128 x 32
    pl->dma = dma_shape && (bf16 ? (pl->w8 && TM == 128 && TN == 128) : (TN != 32 || a.fidx));
    pl->grid = dim3((unsigned)ceil_div(a.M - a.m_lo, TM), (unsigned)ceil_div(a.N, TN), (unsigned)z);
    // selection inside the product: one step on DMA stages, splits of whole
    // regions whose gathered rows fit one table
    if (a.sel_sq) {
        const int R = a.sel_R, S = a.sel_S;
        if (a.idx || !pl->dma || a.steps != 1 || R < 1 || R > 64 || S < 1 || S >= R || a.P < 1 ||
            a.k_chunk > GEMM1_KC_MAX || a.k_chunk % ((long)a.P * (R - S)) != 0 ||
            a.sel_nch < 1 || !a.sel_gc || !a.sel_idx ||
            (((uintptr_t)a.sel_gc) & 15) != 0)
            return hipErrorInvalidValue;
    }
    return hipSuccess;
}

bool gemm1_select_ok(Gemm1Args a, bool bf16) {
    G1Plan pl;
    return a.sel_sq && g1_plan(a, bf16, &pl) == hipSuccess;
}

hipError_t launch_gemm1(Gemm1Args a, bool bf16, hipStream_t s) {
    G1Plan pl;
    const hipError_t e = g1_plan(a, bf16, &pl);
    if (e != hipSuccess)
        return e;
    const int TM = pl.TM, TN = pl.TN;
    const bool vec = pl.vec, w8 = pl.w8, dma = pl.dma;
    const dim3 grid = pl.grid;
    const bool gather = a.idx != nullptr || a.sel_sq != nullptr;
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

} // namespace lstmss
