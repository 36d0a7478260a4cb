// Time-batched weight-gradient MFMA product on the compacted gate gradient
// (kernel template and launcher template; instantiated per storage type in
// wgrad_f32.hip and wgrad_bf16.hip).
//
// Paper: after sparsifying, the kept slices of the gate gradient are a dense
// matrix plus an offset index array, and the weight gradient
// dW[kept rows] += dG_c [x_t; h_{t-1}]^T runs on that matrix (section 3 after
// Fig. 2, section 4).
#pragma once

#include "gemm_common.h"

namespace lstmss {

namespace {

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

// Stages of DMA chunks: bf16 with four row groups per work-group four (three
// chunks in flight: 128 KB dense, 112 KB sparse), other sparse bf16 three
// (chunks two ahead), the rest two.
template <typename TS, bool SPARSE, bool DMA, int NG = WG_NG>
constexpr int wg_stages() {
    return !DMA || sizeof(TS) != 2 ? 2 : NG > WG_NG ? 4 : SPARSE ? 3 : 2;
}
template <typename TS, bool SPARSE, int TT, int ATN, bool VEC, int BC, bool FN = false,
          bool DMA = false, int NG = WG_NG>
__global__ __launch_bounds__(NG * 128, (wg_occupancy<TS, SPARSE, DMA, TT, ATN>())) void wgrad_kernel(WgradArgs a) {
    // NG row groups per work-group, two wavefronts (feature halves) each
    constexpr int NWV = 2 * NG, THREADS = 64 * NWV;  // THREADS shadows the file-wide default
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
    constexpr int gvec = NG * GROWS * cpr, xvec = WG_FEAT * cpr;
    constexpr int RG = (gvec + THREADS - 1) / THREADS;
    constexpr int RX = (xvec + THREADS - 1) / THREADS;
    // two stages: the MFMAs read one while the next batch chunk is written to
    // the other (one barrier per chunk); the kept-slice table is kept per
    // step parity so that a step's routing never races the next step's table
    constexpr int NS = wg_stages<TS, SPARSE, DMA, NG>();
    static_assert(NS <= 3 || !FN, "more than three stages: not the fine structure");
    __shared__ __align__(16) E sX[NS][WG_FEAT][PITCH];
    __shared__ __align__(16) E sG[NS][NG * GROWS][PITCH];
    // kept-slice entries of the steps in flight: sparse DMA chunks copy a
    // step's entries into slot (step mod NSLOT) with its first chunk (at most
    // NS steps are between loaded and routed); otherwise two slots by parity
    constexpr int NSLOT = SPARSE && DMA ? NS : 2;
    __shared__ int sidx[NSLOT][NG][64];

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
    geom(blockIdx.x * NG + gi, r0, rcount, c0, ccount, q0, qcount, j0);
    const int AT = SPARSE ? (rcount + 31) / 32 : 1;
    // compacted-row origin and count of both groups, for the loaders
    int lc0[NG], lcc[NG], lq0[NG], lqc[NG];
#pragma unroll
    for (int k = 0; k < NG; ++k) {
        int t0, t1, t2;
        geom(blockIdx.x * NG + k, t0, t1, lc0[k], lcc[k], lq0[k], lqc[k], t2);
    }

    const int nbc = (B + BC - 1) / BC;
    const int niters = (a.t_end - a.t_begin) * nbc;

    // global -> register staging of one batch chunk; a vector never crosses
    // the end of a row (B is a multiple of VW when VEC).  Each thread's rows
    // are fixed for the whole launch, so their offsets within a step are
    // computed once; a chunk adds the step's base and the batch offset.
    // DMA: instruction k of a chunk fills rows [8k, 8k + 8) of sX (k < 16) or
    // of sG (k >= 16); wavefront w issues k = w, w + NWV, ...
    constexpr int NDI = (WG_FEAT + NG * GROWS) / 8, NDW = NDI / NWV;
    static_assert(!DMA || (NDI % NWV == 0 && WG_FEAT == 128), "DMA instruction split");
    int dofs[DMA ? NDW : 1];
    bool disx[DMA ? NDW : 1];
    if constexpr (DMA) {
#pragma unroll
        for (int i = 0; i < NDW; ++i) {
            const int k = wave + NWV * i;
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
        gok[i] = q < gvec && lr < lcc[k & (NG - 1)];
        gofs[i] = (lc0[k & (NG - 1)] + (gok[i] ? lr : 0)) * B + bb;
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
                const int k = wave + NWV * i;
                const TS *src = k < 16 ? (disx[i] ? xt : ht) + dofs[i] : Gt + dofs[i];
                E *dst = k < 16 ? &sX[lbuf][8 * k][0] : &sG[lbuf][8 * (k - 16)][0];
                dma16(src, (lds_void_t *)dst);
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
        // the step's kept-slice entries, from a clamped (always valid)
        // position: with DMA chunks copied straight into the step's table
        // slot (the routing reads only the group's real entries), else into
        // a register whose entries past the group's count become -1 when
        // stashed, so that nothing waits for this load before then
        if (SPARSE && b0 == 0 && tid < NG * 64) {
            const int k = tid >> 6, e = tid & 63;
            const int32_t *src = a.idx + (long)t * a.kept + (lqc[k] > 0 ? lq0[k] + min(e, lqc[k] - 1) : 0);
            if constexpr (DMA)
                dma4(src, (lds_void_t *)&sidx[tl % NSLOT][k][0]);
            else
                ridx[set] = *src;
        }
        if (FN && b0 == 0 && tid < NG * 64) {  // kept blocks of the group's slice
            const int k = tid >> 6, e = tid & 63;
            const long sl = min((long)blockIdx.x * NG + k, (long)G4 / 32 - 1);
            ridx[set] = a.fidx[((long)t * (G4 / 32) + sl) * a.fkept + min(e, a.fkept - 1)];
        }
    };
    // whether entry e of group k's list at a step is a real entry
    auto entry_ok = [&](int k, int e) {
        if (SPARSE)
            return e < lqc[k];
        return e < a.fkept && (long)blockIdx.x * NG + k < G4 / 32;
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
        if (((SPARSE && !DMA) || FN) && it - tl * nbc == 0 && tid < NG * 64)
            sidx[tl & 1][tid >> 6][tid & 63] = entry_ok(tid >> 6, tid & 63) ? ridx[set] : -1;
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
        // the stored sums are in registers before the loop (the compiler
        // would otherwise keep a full wait for them inside it)
        __builtin_amdgcn_s_waitcnt(0);
    }

    // DMA with NS stages: chunks 0 .. NS - 2 in flight before the loop;
    // wait_chunks(n) waits until at most n chunks' copies are outstanding
    auto wait_chunks = [&](int n) {
        if (NS > 3 && n >= 2)
            __builtin_amdgcn_s_waitcnt(vmcnt_imm((NS > 3 ? 2 : 0) * NDW));
        else if (NS > 2 && n >= 1)
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(NDW));
        else
            __builtin_amdgcn_s_waitcnt(0);
    };
    load(0, 0, 0);
    if (niters > 1 && (!DMA || NS > 2))
        load(1, 1, 1);
    if (DMA && NS > 3 && niters > 2)
        load(2, 0, 2);
    stash(0, 0, 0);
    if (DMA) {
        wait_chunks(min(NS - 2, niters - 1));
        lds_barrier();
    } else {
        __syncthreads();
    }
    constexpr int HALF = BC / 2;
    const int hb = (lane >> 5) * HALF;
    // iteration it computes from LDS buffer it & 1, loads chunk it + 2 into
    // register set it & 1 and stores chunk it + 1 (set and buffer
    // (it + 1) & 1); the loop runs in pairs so that the sets are static
    uint64_t fmask = ~0ull;  // FN: kept blocks of this wavefront's slice at the current step

    // (the lambdas that touch the tile arrays are forced inline: a call would
    // take the arrays' addresses and keep them in scratch memory)
    // sparse routing: csrc[at] is the temporary column (kept row) that
    // accumulator column at * 32 + lane pulls at the current step, -1 if its
    // slice was dropped.  (Routing a step during the next step's first chunk,
    // to overlap the permutes with MFMAs, measured no faster.)
    int csrc[ATN];
    auto lookup = [&](int tl) __attribute__((always_inline)) {
        const int *tab = sidx[SPARSE && DMA ? tl % NSLOT : tl & 1][gi];
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
    // acc[:, at] += tmp routed by csrc (accumulator tiles past the group's
    // rows have src -1 everywhere and stay zero)
    auto route = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int at = 0; at < ATN; ++at) {
            const int src = csrc[at];
            const int saddr = (((src < 0 ? 0 : src) & 31) + (lane & 32)) << 2;
            const int stile = src < 0 ? 0 : (src >> 5);
#pragma unroll
            for (int ft = 0; ft < WG_FT; ++ft) {
                // the permute of each temporary tile, blended by the tile
                // that holds the source (no array indexed by it)
                f32x16 w;
#pragma unroll
                for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const float y = __int_as_float(
                            __builtin_amdgcn_ds_bpermute(saddr, __float_as_int(tmp[ft][tt][v])));
                        w[v] = tt == 0 ? y : (stile == tt ? y : w[v]);
                    }
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    acc[ft][at][v] += src < 0 ? 0.f : w[v];  // dropped: exactly 0, even for inf/NaN
            }
        }
    };

    auto iter = [&](int it, auto sc) __attribute__((always_inline)) {
        constexpr int S0 = decltype(sc)::value, S1 = 1 - S0;
        const int buf = NS == 2 ? S0 : it % NS;
        const int tl = it / nbc, bc = it - tl * nbc;
        if (!DMA && it + 2 < niters)
            load(it + 2, S0, 0);
        // DMA: the next chunk streams into the other buffer (read in the
        // previous iteration), issued once this chunk's operands are in
        // registers (a deeper, three-buffer pipeline measured slower)
        auto issue_next = [&]() {
            if (DMA && it + NS - 1 < niters)
                load(it + NS - 1, NS == 2 ? S1 : S0, (it + NS - 1) % NS);
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
                route();
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
        if (DMA) {
            // chunk it + 1 has landed; chunks it + 2 .. it + NS - 1 may be in flight
            wait_chunks(min(NS - 2, niters - 2 - it));
            lds_barrier();
        } else {
            __syncthreads();
        }
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

// Temporary tiles (kept rows per group / 32) and accumulator tiles (original
// rows per group / 32) of the sparse weight-gradient kernel.  (Grouping four
// regions of 24 kept rows into three exactly filled tiles needs 224
// accumulator registers, one wavefront per SIMD: measured 1.14-1.3x slower
// than the 24-of-32 tiles at 25 % sparsity.)
void wgrad_tiles(int P, int R, int S, int *greg, int *tt, int *at) {
    const int kr = (R - S) * P, rp = R * P;
    *greg = kr <= 32 ? max(1, 32 / kr) : 1;
    *tt = (*greg * kr + 31) / 32;
    *at = (*greg * rp + 31) / 32;
}

// One weight-gradient launch; `dma` takes the LDS-DMA variant (128-byte
// chunks: 32 fp32 or 64 bf16 batch columns).
template <typename TS, bool SP, int TTV, int ATV, bool FN, int NG = WG_NG>
void wg_launch(const WgradArgs &a, bool vec, bool dma, dim3 grid, hipStream_t s) {
    constexpr int DBC = 128 / (int)sizeof(TS);
    if constexpr (NG != WG_NG) {  // other group counts: DMA chunks only
        hipLaunchKernelGGL((wgrad_kernel<TS, SP, TTV, ATV, true, DBC, FN, true, NG>), grid,
                           dim3(NG * 128), 0, s, a);
        return;
    }
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
        // 64-column chunks: bf16 only (fp32 stages 16 or 32 columns)
#define LSTMSS_WG(VE) do { \
        if (a.BC == 16) hipLaunchKernelGGL((wgrad_kernel<TS, SP, TTV, ATV, VE, 16>), grid, dim3(THREADS), 0, s, a); \
        else if (sizeof(TS) == 4 || a.BC == 32) hipLaunchKernelGGL((wgrad_kernel<TS, SP, TTV, ATV, VE, 32>), grid, dim3(THREADS), 0, s, a); \
        else hipLaunchKernelGGL((wgrad_kernel<TS, SP, TTV, ATV, VE, sizeof(TS) == 4 ? 32 : 64>), grid, dim3(THREADS), 0, s, a); } while (0)
        if (vec)
            LSTMSS_WG(true);
        else
            LSTMSS_WG(false);
#undef LSTMSS_WG
    }
}

// --------------------------------------------------------------------------
// bf16 weight gradient with large tiles (DMA chunks of 64 batch columns).
//
// Work-group: 256 original dW rows x 256 features, eight wavefronts of 128
// rows x 64 features (2 x 4 MFMA tiles, accumulated in registers across all
// steps).  Per chunk the staged operands are 256 feature rows and the tile's
// KRT compacted gate-gradient rows; a wavefront reads 0.75 KB of LDS per
// MFMA (the 32-row-group kernel above reads 1.5 KB), and each staged byte
// feeds twice the MFMA work, so fewer chunk copies and reads are waited for
// per MFMA.
// Sparse: the tile covers whole regions (P * R divides 256), so its kept rows
// are the contiguous compacted rows [KRT * tile, KRT * (tile + 1)) at every
// step.  Instead of routing a product of the kept rows, each lane's B operand
// row is, for the step, the compacted row holding its original row or a row
// of zeros in LDS when the row's slice was dropped: the MFMAs run over the
// original rows, a dropped row adding products with zero (twice the MFMAs of
// the kept rows at 50 %, in exchange for no temporary tile and no routing).
// Every row of dW sums its steps from the last down, one MFMA per 16 batch
// columns, in a fixed order (deterministic; the launches of one call continue
// from the stored dW).  Non-finite x or h make a dropped row's product NaN
// (0 * inf), where the routing kernel adds nothing.
// --------------------------------------------------------------------------
constexpr int WB_ROWS = 256, WB_FEAT = 256, WB_THREADS = 512;

template <int KRT>
constexpr int wb_stages() { return KRT <= 128 ? 3 : 2; }

template <int KRT, bool SP>
__global__ __launch_bounds__(WB_THREADS, 2) void wgrad_big_kernel(WgradArgs a) {
    constexpr int NS = wb_stages<KRT>();
    constexpr int NDI = (WB_FEAT + KRT) / 8;      // 1 KB copies per chunk
    constexpr int NDW = NDI / 8;                  // per wavefront
    static_assert(NDI % 8 == 0 && KRT % 64 == 0, "whole copies per wavefront");
    constexpr int NQ = SP ? KRT : 1;              // kept-slice entries per step (at most KRT / P)
    __shared__ __align__(16) uint16_t sX[NS][WB_FEAT][64];
    __shared__ __align__(16) uint16_t sG[NS][KRT + 1][64];  // row KRT: zeros
    __shared__ int sidx[SP ? NS : 1][NQ];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: descriptors stay scalar
    const int rh = wave & 1, fq = wave >> 1;      // row half, feature quarter
    const int I = a.I, H = a.H, B = a.B;
    const int NC = I + H, G4 = 4 * H;
    const int r0 = blockIdx.x * WB_ROWS, n0 = blockIdx.y * WB_FEAT;
    const bf16_t *Gc = (const bf16_t *)a.Gc;
    const bf16_t *x = (const bf16_t *)a.x;
    const bf16_t *h = (const bf16_t *)a.h;
    // sparse geometry: regions of the tile, their kept-slice entries and rows
    const int ks = SP ? a.R - a.S : 0;
    const int rpw = SP ? WB_ROWS / (a.P * a.R) : 0;
    const int q0 = blockIdx.x * rpw * ks;         // first kept-slice entry
    const int c0 = SP ? blockIdx.x * KRT : r0;    // first compacted row
    const int nq = rpw * ks;                      // entries of the tile (<= NQ)

    if (tid < NS * 8)
        *(u16x8 *)&sG[tid >> 3][KRT][8 * (tid & 7)] = u16x8{0, 0, 0, 0, 0, 0, 0, 0};

    // copies: instruction k fills 8 rows of sX (k < 32) or sG; wavefront w
    // issues k = w, w + 8, ...; lane j fills 16-byte piece j & 7 of row j >> 3.
    // Byte offsets within a step's operand (x or h by the instruction's
    // first feature, all 8 rows on the same side since I % 8 == 0)
    int voff[NDW];
#pragma unroll
    for (int i = 0; i < NDW; ++i) {
        const int k = wave + 8 * i;
        const int rr = 8 * (k < 32 ? k : k - 32) + (lane >> 3);
        const int pc = (lane & 7) ^ wg_swz(rr);
        if (k < 32) {
            const int n = min(n0 + rr, NC - 1);
            voff[i] = 2 * ((n < I ? n : n - I) * B + pc * 8);
        } else {
            voff[i] = 2 * (min(c0 + rr, a.Kp - 1) * B + pc * 8);
        }
    }
    const int nbc = B / 64;
    const int niters = (a.t_end - a.t_begin) * nbc;
    auto load = [&](int it) __attribute__((always_inline)) {
        const int tl = it / nbc, b0 = (it - tl * nbc) * 64;
        const int t = a.t_end - 1 - tl;
        const int buf = it % NS;
        const i32x4 rx = buf_rsrc(x + (long)t * I * B, 2u * I * B);
        const i32x4 rhh = buf_rsrc(h + (long)t * H * B, 2u * H * B);
        const i32x4 rg = buf_rsrc(Gc + (long)t * a.Kp * B, 2u * a.Kp * B);
#pragma unroll
        for (int i = 0; i < NDW; ++i) {
            const int k = wave + 8 * i;
            if (k < 32)
                dma16_buf(n0 + 8 * k < I ? rx : rhh, voff[i], 2 * b0, (lds_void_t *)&sX[buf][8 * k][0]);
            else
                dma16_buf(rg, voff[i], 2 * b0, (lds_void_t *)&sG[buf][8 * (k - 32)][0]);
        }
        if constexpr (SP) {
            // the step's kept-slice entries of the tile's regions, with its first chunk
            if (b0 == 0 && wave * 64 < nq) {
                const int e = min(q0 + wave * 64 + lane, a.kept - 1);
                dma4(a.idx + (long)t * a.kept + e, (lds_void_t *)&sidx[tl % NS][wave * 64]);
            }
        }
    };
    auto wait_chunks = [&](int n) {
        if (NS > 2 && n >= 2)
            __builtin_amdgcn_s_waitcnt(vmcnt_imm((NS > 2 ? 2 : 0) * NDW));
        else if (n >= 1)
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(NDW));
        else
            __builtin_amdgcn_s_waitcnt(0);
    };

    f32x16 acc[2][4];
#pragma unroll
    for (int ft = 0; ft < 2; ++ft)
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                acc[ft][rt][v] = 0.f;
    // accumulator tile (ft, rt): column = dW row r0 + rh * 128 + rt * 32 +
    // lane % 32, register v = feature n0 + fq * 64 + ft * 32 + acc_row(lane, v)
    if (a.accumulate) {
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
            const int row = r0 + rh * 128 + rt * 32 + (lane & 31);
            if (row >= G4)
                continue;
            const float *src = a.dW + (long)row * NC;
#pragma unroll
            for (int ft = 0; ft < 2; ++ft)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int f = n0 + fq * 64 + ft * 32 + acc_row(lane, v);
                    if (f < NC)
                        acc[ft][rt][v] = src[f];
                }
        }
        __builtin_amdgcn_s_waitcnt(0);
    }

    // every buffer in flight before the loop: chunks 0 .. NS - 1
#pragma unroll
    for (int c = 0; c < NS; ++c)
        if (c < niters)
            load(c);

    // LDS element offsets of this lane's operand rows (A: features, fixed;
    // B: the step's row map) and their piece permutation
    const int hp = (lane >> 5) * 4;               // first 16-byte piece of this half
    int aoff[2], asw[2], boff[4], bsw[4];
#pragma unroll
    for (int ft = 0; ft < 2; ++ft) {
        const int f = fq * 64 + ft * 32 + (lane & 31);
        aoff[ft] = f * 64;
        asw[ft] = wg_swz(f);
    }
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
        const int slot = rh * 128 + rt * 32 + (lane & 31);
        boff[rt] = slot * 64;
        bsw[rt] = wg_swz(slot);
    }
    // the row map of step tl (sparse): the compacted row holding each of this
    // lane's original rows at that step, or the zero row
    auto row_map = [&](int tl) __attribute__((always_inline)) {
        if constexpr (SP) {
            const int *tab = sidx[tl % NS];
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) {
                const int r = r0 + rh * 128 + rt * 32 + (lane & 31);
                int slot = KRT;
                if (r < G4) {
                    const int js = r / a.P, reg = js / a.R;
                    const int e0 = reg * ks, e1 = min(e0 + ks, a.kept);
                    for (int e = e0; e < e1; ++e)
                        if (tab[e - q0] == js)
                            slot = e * a.P + (r - js * a.P) - c0;
                }
                boff[rt] = slot * 64;
                bsw[rt] = wg_swz(slot);
            }
        }
    };
    // operands of k-step s (16 batch columns: 8 per lane half) of buffer buf
    // into register set st
    u16x8 fa[2][2], fb[2][4];
    auto rd = [&](int buf, int s, auto setc) __attribute__((always_inline)) {
        constexpr int st = decltype(setc)::value;
        const uint16_t *xb = &sX[buf][0][0];
        const uint16_t *gb = &sG[buf][0][0];
#pragma unroll
        for (int ft = 0; ft < 2; ++ft)
            fa[st][ft] = *(const u16x8 *)(xb + aoff[ft] + (((hp + s) ^ asw[ft]) << 3));
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
            fb[st][rt] = *(const u16x8 *)(gb + boff[rt] + (((hp + s) ^ bsw[rt]) << 3));
    };
    // (the scheduler keeps each group in place: reading the next operands
    // into a set ahead of the MFMAs that still use it costs registers)
    auto mma = [&](auto setc) __attribute__((always_inline)) {
        constexpr int st = decltype(setc)::value;
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ft = 0; ft < 2; ++ft)
#pragma unroll
            for (int rt = 0; rt < 4; ++rt)
                acc[ft][rt] = mfma32x32x16bf(fa[st][ft], fb[st][rt], acc[ft][rt]);
        __builtin_amdgcn_sched_barrier(0);
    };
    constexpr std::integral_constant<int, 0> S0{};
    constexpr std::integral_constant<int, 1> S1{};

    if (niters > 0) {
        wait_chunks(min(NS - 1, niters - 1));
        lds_barrier();
        row_map(0);
        rd(0, 0, S0);
        rd(0, 1, S1);
    }
    // Iteration it multiplies chunk it (k-steps 0 and 1 already in registers)
    // and, between its last two k-steps, meets the other wavefronts once
    // chunk it + 1 has landed: chunk it's buffer then takes chunk it + NS, and
    // the first k-steps of chunk it + 1 are read while the last MFMAs run.
    for (int it = 0; it + 1 < niters; ++it) {
        const int buf = it % NS;
        mma(S0);
        rd(buf, 2, S0);
        mma(S1);
        rd(buf, 3, S1);
        mma(S0);
        // chunk it + 1 has landed; chunks it + 2 .. it + NS - 1 may be in flight
        wait_chunks(min(NS - 2, niters - 2 - it));
        lds_barrier();
        if (it + NS < niters)
            load(it + NS);
        const int nb = (it + 1) % NS;
        if ((it + 1) % nbc == 0)
            row_map((it + 1) / nbc);
        rd(nb, 0, S0);
        mma(S1);
        rd(nb, 1, S1);
    }
    if (niters > 0) {  // the last chunk
        const int buf = (niters - 1) % NS;
        mma(S0);
        rd(buf, 2, S0);
        mma(S1);
        rd(buf, 3, S1);
        mma(S0);
        mma(S1);
    }

#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
        const int row = r0 + rh * 128 + rt * 32 + (lane & 31);
        if (row >= G4)
            continue;
        float *dst = a.dW + (long)row * NC;
#pragma unroll
        for (int ft = 0; ft < 2; ++ft)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int f = n0 + fq * 64 + ft * 32 + acc_row(lane, v);
                if (f < NC)
                    dst[f] = acc[ft][rt][v];
            }
    }
}

// The large-tile bf16 kernel for this call, if its conditions hold: DMA
// chunks, I a multiple of 8, the dense product or a coarse structure whose
// regions tile 256 rows and keep 128 or 192 of them per tile.  Returns false
// otherwise (the caller launches the routing kernel).
bool wgrad_big_launch(const WgradArgs &a, bool sparse, hipStream_t s) {
    // per-step operands addressed with 32-bit byte offsets; x / h chosen per
    // 8 feature rows
    if (a.I % 8 != 0 || 2L * a.Kp * a.B >= (1L << 31) || 2L * a.I * a.B >= (1L << 31) ||
        2L * a.H * a.B >= (1L << 31))
        return false;
    // sparsity 0 keeps every slice in order: the dense product, bit for bit
    if (sparse && a.S == 0)
        sparse = false;
    int krt = WB_ROWS;
    if (sparse) {
        const int pr = a.P * a.R;
        if (pr <= 0 || pr > WB_ROWS || WB_ROWS % pr != 0 || a.S >= a.R)
            return false;
        krt = WB_ROWS / a.R * (a.R - a.S);
        if (WB_ROWS % a.R != 0 || krt % 64 != 0)
            return false;
    }
    dim3 grid((unsigned)ceil_div(4L * a.H, WB_ROWS), (unsigned)ceil_div(a.I + a.H, WB_FEAT));
    // sparse: the zero rows' MFMAs cost more than the routing kernel's
    // permutes below half the rows kept (75 % sparsity: 1.88 vs 1.67 ms at
    // H = 4096, B = 256, T = 25), and with fewer tiles than CUs the routing
    // kernel's smaller tiles fill the GPU better (H = 1024, B = 64)
    if (sparse && (krt < WB_ROWS / 2 || (long)grid.x * grid.y < 256))
        return false;
    if (!sparse)
        hipLaunchKernelGGL((wgrad_big_kernel<256, false>), grid, dim3(WB_THREADS), 0, s, a);
    else if (krt == 192)
        hipLaunchKernelGGL((wgrad_big_kernel<192, true>), grid, dim3(WB_THREADS), 0, s, a);
    else if (krt == 128)
        hipLaunchKernelGGL((wgrad_big_kernel<128, true>), grid, dim3(WB_THREADS), 0, s, a);
    else if (krt == 64)
        hipLaunchKernelGGL((wgrad_big_kernel<64, true>), grid, dim3(WB_THREADS), 0, s, a);
    else
        return false;
    return true;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }

// One weight-gradient call in storage type TS (the instantiations live in
// wgrad_f32.hip and wgrad_bf16.hip, so that the two compile in parallel).
template <typename TS>
hipError_t launch_wgrad_t(WgradArgs a, bool sparse, hipStream_t s) {
    constexpr bool bf16 = sizeof(TS) == 2;
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
        wg_launch<TS, false, 1, 1, true>(a, vec, bf16 ? false : dma_ok(32), grid, s);
        return hipGetLastError();
    }
    if constexpr (bf16) {
        if (a.big && dma_ok(64) && wgrad_big_launch(a, sparse, s))
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
    // bf16 with DMA chunks: four row groups per work-group of eight wavefronts
    // (one per CU), so that every staged feature row feeds twice the kept
    // rows: the bf16 MFMAs outrun the rate the stages reach LDS
    const bool ng4 = bf16 && dma && (!sparse || (tt == 1 && at <= 2));
    const int ng = ng4 ? 4 : WG_NG;
    dim3 grid((unsigned)ceil_div(groups, ng), (unsigned)ceil_div(a.I + a.H, WG_FEAT));
#define LSTMSS_WGA(TTV) do { \
        if (at <= 1) { if (TTV == 1 && ng4) wg_launch<TS, true, TTV, 1, false, TTV == 1 ? 4 : WG_NG>(a, vec, dma, grid, s); \
                       else wg_launch<TS, true, TTV, 1, false>(a, vec, dma, grid, s); } \
        else if (at <= 2) { if (TTV == 1 && ng4) wg_launch<TS, true, TTV, 2, false, TTV == 1 ? 4 : WG_NG>(a, vec, dma, grid, s); \
                            else wg_launch<TS, true, TTV, 2, false>(a, vec, dma, grid, s); } \
        else wg_launch<TS, true, TTV, 4, false>(a, vec, dma, grid, s); } while (0)
    if (!sparse) { if (ng4) wg_launch<TS, false, 1, 1, false, 4>(a, vec, dma, grid, s);
                   else wg_launch<TS, false, 1, 1, false>(a, vec, dma, grid, s); }
    else if (tt == 1) LSTMSS_WGA(1);
    else LSTMSS_WGA(2);
#undef LSTMSS_WGA
    return hipGetLastError();
}

} // namespace

} // namespace lstmss
