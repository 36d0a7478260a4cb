// Backward elementwise gate-gradient kernel fused with structural
// sparsifying (score, per-region selection, compaction), plus the small
// helper kernels of the backward driver.
//
// Paper: section 3 (coarse-grained structural sparsifying of the gate
// gradient dnet, offset index array of the kept slices); the gate-gradient
// data flow is the one of Fig. 1 for the standard LSTM cell.
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "select.h"

namespace lstmss {

namespace {

constexpr int CELL_THREADS = 512;

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
    const float dh = sum_parts(a.dH_up[e], a.dh_part + e, a.dh_nparts, a.dh_stride);
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

template <typename TS, int MODE>
__global__ __launch_bounds__(CELL_THREADS) void cell_select_kernel(CellArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int NW = CELL_THREADS / 64;
    const int B = a.B, P = a.P, R = a.R;
    const long G = 4L * a.H;

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

    // Phase 1b: per-row sum of squares in the fixed order (each 64-column
    // chunk combined by index xor 32, 16, ..., 1, chunks added in order).
    // With B <= 2^k < 64 every square at index >= 2^k is zero and adding it is
    // exact, so 2^k lanes per row give the same value; a wavefront then
    // handles 64 / 2^k rows at once.  Row sums for the bias gradient ride
    // along.
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
            for (int c = 0; 64 * c < B; ++c) {  // chunks of 64 batch columns
                const int b = 64 * c + sl;
                const float v = (lr < nrows && b < B) ? sdG[lr * B + b] : 0.f;
                rsum += v;
                if (MODE != CELL_DENSE) {
                    double q = (double)v * (double)v;
                    for (int off = lpr >> 1; off >= 1; off >>= 1)
                        q = q + shfl_xor_f64(q, off);
                    part = c == 0 ? q : part + q;
                }
            }
            for (int off = lpr >> 1; off >= 1; off >>= 1)
                rsum += shfl_xor_f32(rsum, off);
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

// Lane i receives lane i + N of its 16-lane row (a DPP row shift; lanes
// whose source leaves the row receive 0).  Used for the steps off = 8, 4, 2,
// 1 of a butterfly (each lane adds the value of lane i ^ off to its own):
// the lanes that feed the first lane of an aligned group of 2 off lanes have
// i ^ off = i + off, so that first lane gets the butterfly's bits.
template <int N>
__device__ __forceinline__ float row_down_f32(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x100 + N, 0xf, 0xf, true));
}
template <int N>
__device__ __forceinline__ double row_down_f64(double v) {
    const long long x = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(x & 0xffffffffLL), 0x100 + N, 0xf, 0xf, true);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(x >> 32), 0x100 + N, 0xf, 0xf, true);
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// Lane i receives lane i ^ 32 (X = 32) or lane i ^ 16 (X = 16): the swap of
// the two halves of the wavefront, or of its odd and even 16-lane rows.
template <int X>
__device__ __forceinline__ unsigned lane_xor_swap(unsigned v) {
    static_assert(X == 16 || X == 32, "16 or 32");
    const int lane = threadIdx.x & 63;
    if (X == 32) {
        const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        return lane < 32 ? r[1] : r[0];
    } else {
        const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        return (lane & 16) ? r[0] : r[1];
    }
}
template <int X>
__device__ __forceinline__ float lane_xor_f32(float v) {
    return __uint_as_float(lane_xor_swap<X>(__float_as_uint(v)));
}

template <int X>
__device__ __forceinline__ double lane_xor_f64(double v) {
    const long long x = __double_as_longlong(v);
    const unsigned lo = lane_xor_swap<X>((unsigned)(x & 0xffffffffLL));
    const unsigned hi = lane_xor_swap<X>((unsigned)((unsigned long long)x >> 32));
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Step OFF of a 64-lane butterfly, for the lanes that feed lane 0 (and the
// first lane of every aligned group of 2 OFF lanes): the value of lane
// i ^ OFF, moved by lane swaps (OFF = 32, 16) or DPP row shifts (OFF <= 8).
template <int OFF>
__device__ __forceinline__ float bfly_f32(float v) {
    if constexpr (OFF >= 16)
        return lane_xor_f32<OFF>(v);
    else
        return row_down_f32<OFF>(v);
}
template <int OFF>
__device__ __forceinline__ double bfly_f64(double v) {
    if constexpr (OFF >= 16)
        return lane_xor_f64<OFF>(v);
    else
        return row_down_f64<OFF>(v);
}

// The sum a W-lane xor butterfly (offsets W / 2, ..., 1) leaves in the first
// lane of every aligned group of W lanes (the other lanes hold partial sums).
template <int W>
__device__ __forceinline__ double lead_sum_f64(double v) {
    if constexpr (W >= 64)
        v = v + bfly_f64<32>(v);
    if constexpr (W >= 32)
        v = v + bfly_f64<16>(v);
    if constexpr (W >= 16)
        v = v + bfly_f64<8>(v);
    if constexpr (W >= 8)
        v = v + bfly_f64<4>(v);
    if constexpr (W >= 4)
        v = v + bfly_f64<2>(v);
    if constexpr (W >= 2)
        v = v + bfly_f64<1>(v);
    return v;
}
template <int W>
__device__ __forceinline__ float lead_sum_f32(float v) {
    if constexpr (W >= 64)
        v = v + bfly_f32<32>(v);
    if constexpr (W >= 32)
        v = v + bfly_f32<16>(v);
    if constexpr (W >= 16)
        v = v + bfly_f32<8>(v);
    if constexpr (W >= 8)
        v = v + bfly_f32<4>(v);
    if constexpr (W >= 4)
        v = v + bfly_f32<2>(v);
    if constexpr (W >= 2)
        v = v + bfly_f32<1>(v);
    return v;
}

// ---------------------------------------------------------------------------
// Register-resident variant for small work-groups (<= 32 rows, <= 32 slices,
// B <= 256): a row is owned by LPR lanes (the next power of two >= B, at most
// 64), lane l holding batch columns l, l+64, ... (one per 64-column chunk);
// with B <= LPR < 64 the squares at index >= LPR are zero, so an LPR-lane
// butterfly gives the fixed score order exactly.  Values stay in registers from the gate-gradient
// formula to the compacted store; one wavefront scores, selects (ballot
// prefix within each region) and places the slices.
// ---------------------------------------------------------------------------
constexpr int RK_WAVES = 8;

template <typename TS, int MODE, int LPR, int NJ>
__global__ __launch_bounds__(RK_WAVES * 64) void cell_rows_kernel(CellArgs a) {
    constexpr int RPW = 64 / LPR;                       // rows per wavefront pass
    constexpr int NP = (32 + RK_WAVES * RPW - 1) / (RK_WAVES * RPW);
    __shared__ double srowsq[32];
    __shared__ int sslot[32];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int B = a.B, H = a.H, P = a.P, R = a.R;
    const long spw = (long)a.regions_per_wg * R;
    const long j0 = blockIdx.x * spw;
    const int nsl = (int)min(spw, a.nslices - j0);
    const int row0 = (int)(j0 * P);
    const int nrows = nsl * P;
    const int sub = lane / LPR, sl = lane - sub * LPR;

    const TS *__restrict__ gates = (const TS *)a.gates;
    const float *__restrict__ dHup = a.dH_up;
    const float *__restrict__ ct = a.c_t;
    const float *__restrict__ cp = a.c_prev;
    const float *__restrict__ dcin = a.dc_in;
    TS *dGc = (TS *)a.dGc;
    TS *dbg = (TS *)a.dbg;

    // Phase 1: loads of every owned element first, then the formulas.
    float v[NP][NJ];
    float l_dh[NP][NJ], l_o[NP][NJ], l_a[NP][NJ], l_b[NP][NJ], l_ct[NP][NJ], l_x[NP][NJ];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        const int lr = (p * RK_WAVES + wave) * RPW + sub;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int b = sl + 64 * j;
            const bool in = lr < nrows && b < B;
            const int r = row0 + (in ? lr : 0);
            const int g = r / H, u = r - g * H;
            const int e = u * B + (in ? b : 0);
            if (MODE == CELL_GIVEN) {
                l_x[p][j] = in ? st<TS>::load((const TS *)a.dG_in, (long)r * B + b) : 0.f;
                continue;
            }
            l_dh[p][j] = in ? sum_parts(dHup[e], a.dh_part + e, a.dh_nparts, a.dh_stride) : 0.f;
            l_ct[p][j] = in ? ct[e] : 0.f;
            l_o[p][j] = in ? st<TS>::load(gates, (long)(3 * H + u) * B + b) : 0.f;
            // gate-specific operands: i rows need (i, g), f rows (f, c_{t-1}),
            // g rows (i, g); all but o rows need dc_t
            const int ga = g == 1 ? 1 : 0, gb = 2;
            l_a[p][j] = (in && g < 3) ? st<TS>::load(gates, (long)(ga * H + u) * B + b) : 0.f;
            l_b[p][j] = (in && g < 3) ? (g == 1 ? cp[e] : st<TS>::load(gates, (long)(gb * H + u) * B + b)) : 0.f;
            l_x[p][j] = (in && g < 3 && dcin) ? dcin[e] : 0.f;
        }
    }
    double part[NP];
    float rsum[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        const int lr = (p * RK_WAVES + wave) * RPW + sub;
        part[p] = 0.0;
        rsum[p] = 0.f;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int b = sl + 64 * j;
            const bool in = lr < nrows && b < B;
            float val;
            if (MODE == CELL_GIVEN) {
                val = l_x[p][j];
            } else {
                const int r = row0 + (in ? lr : 0);
                const int g = r / H, u = r - g * H;
                const float dh = l_dh[p][j], tc = tanhf(l_ct[p][j]), o = l_o[p][j];
                if (g == 3) {
                    val = dh * tc * o * (1.f - o);
                } else {
                    const float dcv = l_x[p][j] + dh * o * (1.f - tc * tc);
                    if (g == 1) {
                        const float f = l_a[p][j];
                        if (in)
                            a.dc_out[u * B + b] = dcv * f;
                        val = dcv * l_b[p][j] * f * (1.f - f);
                    } else {
                        const float i = l_a[p][j], gg = l_b[p][j];
                        val = g == 0 ? dcv * gg * i * (1.f - i) : dcv * i * (1.f - gg * gg);
                    }
                }
                val = st<TS>::rnd(val);
                if (in && dbg)
                    st<TS>::store(dbg, (long)r * B + b, val);
                if (in && MODE == CELL_DENSE)
                    st<TS>::store(dGc, (long)r * B + b, val);
            }
            val = in ? val : 0.f;
            v[p][j] = val;
            rsum[p] += val;
            if (MODE != CELL_DENSE) {
                // chunk j of the row: the LPR-lane butterfly's sum in the
                // row's first lane, then fold into the row
                const double q = lead_sum_f64<LPR>((double)val * (double)val);
                part[p] = j == 0 ? q : part[p] + q;
            }
        }
        rsum[p] = lead_sum_f32<LPR>(rsum[p]);  // used by the row's first lane
        if (sl == 0 && lr < nrows) {
            if (MODE == CELL_DENSE) {
                if (a.db)
                    a.db[row0 + lr] += rsum[p];
            } else {
                srowsq[lr] = part[p];
            }
        }
    }
    if (MODE == CELL_DENSE)
        return;
    __syncthreads();

    // Phases 2-4 in wavefront 0: lane j scores slice j, counts the slices of
    // its region that outrank it, and takes its slot from a ballot prefix.
    if (wave == 0) {
        const int j = lane;
        const bool valid = j < nsl;
        double sc = 0.0;
        if (valid) {
            sc = srowsq[j * P];
            for (int p = 1; p < P; ++p)
                sc = sc + srowsq[j * P + p];
            if (a.scores)
                a.scores[j0 + j] = sc;
        }
        const SliceSel sel = rank_slices(sc, j0, nsl, R, a.S, a.nslices);
        if (sel.slot >= 0)
            a.idx[sel.slot] = (int32_t)(j0 + j);
        if (valid)
            sslot[j] = sel.slot;
    }
    __syncthreads();

    // Phase 5: kept values from registers to the compacted matrix; bias.
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        const int lr = (p * RK_WAVES + wave) * RPW + sub;
        if (lr >= nrows)
            continue;
        const int slot = sslot[lr / P];
        if (slot < 0)
            continue;
        const long crow = (long)slot * P + lr % P;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int b = sl + 64 * j;
            if (b < B)
                st<TS>::store(dGc, crow * B + b, v[p][j]);
        }
        if (sl == 0 && a.db)
            a.db[row0 + lr] += rsum[p];
    }
}

// ---------------------------------------------------------------------------
// Split variant for large shapes, two kernels per step.
//
// cell_elem_kernel: element-parallel over (4 units x one 64-column batch
// chunk) per work-group, one unit per wavefront, lane l holding batch column
// 64c + l, so every CU has loads in flight.  Each (unit, batch) element is
// loaded once and gives all four gate gradients.  It writes the gate
// gradient (straight to the compacted matrix when nothing is dropped, else to
// a staging matrix), dc_{t-1}, and per (row, chunk) the fp64 chunk sum of
// squares (fixed 64-lane butterfly) and the fp32 row sum.  MODE CELL_GIVEN
// reads the four rows of each unit from a given gate-gradient matrix instead
// (the standalone selection) and writes only the chunk sums of squares; the
// given matrix is then the select kernel's staging matrix.
//
// cell_select_kernel2: one work-group per group of regions folds the chunk
// sums of its rows in order, scores and selects the slices (one wavefront),
// and copies the kept rows from the staging matrix.
// ---------------------------------------------------------------------------
constexpr int EK_UNITS = 4;
constexpr int EK_WAVES = 4;

// FBLK (dense mode, the fine structure with 32-row slices): instead of the
// chunk row sums, each row's per-block sums of squares (fp64, the My-lane
// butterfly of the block's squares) and sums (fp32, the same butterfly of its
// values) go to blk_sq / blk_rs [4H][nb], from each block's first lane.
template <typename TS, int MODE, bool FBLK = false>
__global__ __launch_bounds__(EK_WAVES * 64) void cell_elem_kernel(CellArgs a) {
    static_assert(!FBLK || MODE == CELL_DENSE, "block sums: dense mode");
    constexpr bool SPARSE = MODE != CELL_DENSE, GIVEN = MODE == CELL_GIVEN;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int B = a.B, H = a.H;
    const int c = blockIdx.y, nch = gridDim.y;
    const int b = 64 * c + lane;
    const bool bin = b < B;
    const TS *__restrict__ gates = (const TS *)a.gates;
    const float *__restrict__ dHup = a.dH_up;
    const float *__restrict__ ct = a.c_t;
    const float *__restrict__ cp = a.c_prev;
    const float *__restrict__ dcin = a.dc_in;
    constexpr int UPW = EK_UNITS / EK_WAVES;
    float lg[UPW][4], ldh[UPW], lct[UPW], lcp[UPW], ldc[UPW];
    int uu[UPW];
    bool ok[UPW];
#pragma unroll
    for (int k = 0; k < UPW; ++k) {
        const int u = blockIdx.x * EK_UNITS + wave * UPW + k;
        uu[k] = u;
        ok[k] = u < H && bin;
        const int e = (u < H ? u : 0) * B + (bin ? b : 0);
        if (GIVEN) {  // the unit's four rows of the given matrix
#pragma unroll
            for (int g = 0; g < 4; ++g)
                lg[k][g] = ok[k] ? st<TS>::load((const TS *)a.dG_in, (long)(g * H + u) * B + b) : 0.f;
            continue;
        }
#pragma unroll
        for (int g = 0; g < 4; ++g)
            lg[k][g] = ok[k] ? st<TS>::load(gates, (long)(g * H + u) * B + b) : 0.f;
        lct[k] = ok[k] ? ct[e] : 0.f;
        lcp[k] = ok[k] ? cp[e] : 0.f;
        ldc[k] = (ok[k] && dcin) ? dcin[e] : 0.f;
        ldh[k] = ok[k] ? sum_parts<16>(dHup[e], a.dh_part + e, a.dh_nparts, a.dh_stride) : 0.f;
    }
    TS *out = (TS *)(SPARSE ? a.stage : a.dGc);
    TS *dbg = (TS *)a.dbg;
#pragma unroll
    for (int k = 0; k < UPW; ++k) {
        const int u = uu[k];
        float v[4];
        if (GIVEN) {
#pragma unroll
            for (int g = 0; g < 4; ++g)
                v[g] = lg[k][g];
        } else {
            const float ig = lg[k][0], fg = lg[k][1], gg = lg[k][2], og = lg[k][3];
            const float tc = tanhf(lct[k]);
            const float dcv = ldc[k] + ldh[k] * og * (1.f - tc * tc);
            v[0] = st<TS>::rnd(dcv * gg * ig * (1.f - ig));
            v[1] = st<TS>::rnd(dcv * lcp[k] * fg * (1.f - fg));
            v[2] = st<TS>::rnd(dcv * ig * (1.f - gg * gg));
            v[3] = st<TS>::rnd(ldh[k] * tc * og * (1.f - og));
            if (ok[k])
                a.dc_out[u * B + b] = dcv * fg;
        }
        if (ok[k] && !GIVEN) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const long r = (long)g * H + u;
                st<TS>::store(out, r * B + b, v[g]);
                if (dbg)
                    st<TS>::store(dbg, r * B + b, v[g]);
            }
        }
        if constexpr (FBLK) {
            double q[4];
            float rs[4];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const float x = ok[k] ? v[g] : 0.f;
                q[g] = (double)x * (double)x;
                rs[g] = x;
            }
            auto sums = [&](auto w) {
                constexpr int W = decltype(w)::value;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    q[g] = lead_sum_f64<W>(q[g]);
                    rs[g] = lead_sum_f32<W>(rs[g]);
                }
            };
            const int My = a.My, nb = a.nb;
            switch (My) {
            case 2: sums(std::integral_constant<int, 2>()); break;
            case 4: sums(std::integral_constant<int, 4>()); break;
            case 8: sums(std::integral_constant<int, 8>()); break;
            case 16: sums(std::integral_constant<int, 16>()); break;
            case 32: sums(std::integral_constant<int, 32>()); break;
            default: sums(std::integral_constant<int, 64>()); break;
            }
            const int bi = (64 * c + lane) >> __builtin_ctz(My);
            if ((lane & (My - 1)) == 0 && bi < nb && u < H) {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const long r = (long)g * H + u;
                    a.blk_sq[r * nb + bi] = q[g];
                    a.blk_rs[r * nb + bi] = rs[g];
                }
            }
            continue;
        }
        // per row the 64-lane butterflies' sums (lane 0's bits)
        double q[4];
        float rs[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const float x = ok[k] ? v[g] : 0.f;
            q[g] = (double)x * (double)x;
            rs[g] = x;
        }
#define LSTMSS_EK_STEP(O)                                                                          \
    _Pragma("unroll") for (int g = 0; g < 4; ++g) {                                               \
        if (SPARSE)                                                                               \
            q[g] = q[g] + bfly_f64<O>(q[g]);                                                      \
        if (!GIVEN)                                                                               \
            rs[g] = rs[g] + bfly_f32<O>(rs[g]);                                                   \
    }
        LSTMSS_EK_STEP(32) LSTMSS_EK_STEP(16) LSTMSS_EK_STEP(8)
        LSTMSS_EK_STEP(4) LSTMSS_EK_STEP(2) LSTMSS_EK_STEP(1)
#undef LSTMSS_EK_STEP
        if (lane == 0 && u < H) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const long r = (long)g * H + u;
                if (SPARSE)
                    a.chunk_sq[r * nch + c] = q[g];
                if (!GIVEN)
                    a.chunk_rs[r * nch + c] = rs[g];
            }
        }
    }
}

// One wavefront per group of regions_per_wg * R slices (<= 64 slices, <= 256
// rows), one wavefront per work-group so that the groups spread over the CUs:
// fold the chunk sums of each row in order, score the slices, rank each
// slice against the R slices of its region, and copy the kept rows.
template <typename TS>
__global__ __launch_bounds__(64) void cell_select_kernel2(CellArgs a) {
    __shared__ int sslot[64];
    __shared__ int sinv[64];  // kept slice (local index) of each local slot
    __shared__ int s_nkept;
    const int lane = threadIdx.x;
    const int B = a.B, P = a.P, R = a.R;
    const int nch = (B + 63) / 64;
    const long spw = (long)a.regions_per_wg * R;
    const long j0 = blockIdx.x * spw;
    const int nsl = (int)min(spw, a.nslices - j0);
    const long row0 = j0 * P;
    const int nrows = nsl * P;
    const SliceSel sel = select_slices(a.chunk_sq, nch, j0, nsl, P, R, a.S, a.nslices);
    const int j = lane;
    if (j < nsl && a.scores)
        a.scores[j0 + j] = sel.score;
    // the group's kept slices fill a contiguous run of slots from slot0
    // (regions start at multiples of R, each region's slots at R - S times
    // its number)
    const long slot0 = (j0 / R) * (R - a.S);
    if (sel.slot >= 0) {
        a.idx[sel.slot] = (int32_t)(j0 + j);
        sinv[sel.slot - slot0] = j;
    }
    if (j < nsl)
        sslot[j] = sel.slot;
    if (lane == 0)
        s_nkept = sel.nkept;
    __syncthreads();
    // copy the kept rows into their contiguous slots: lanes over the
    // destination's 16-byte vectors, eight loads in flight before their
    // stores
    const int rowbytes = B * (int)sizeof(TS);
    if ((rowbytes & 15) == 0) {
        const int rv = rowbytes / 16, sv = P * rv;  // vectors per row / per slice
        const uint4 *__restrict__ src = (const uint4 *)a.stage + row0 * rv;
        uint4 *__restrict__ dst = (uint4 *)a.dGc + slot0 * sv;
        const int nv = s_nkept * sv;
        for (int v0 = 0; v0 < nv; v0 += 8 * 64) {
            uint4 buf[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int v = v0 + u * 64 + lane;
                uint4 x = make_uint4(0, 0, 0, 0);
                if (v < nv) {
                    const int q = v / sv, r = v - q * sv;  // local slot, vector within it
                    x = src[(long)sinv[q] * sv + r];
                }
                buf[u] = x;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int v = v0 + u * 64 + lane;
                if (v < nv)
                    dst[v] = buf[u];
            }
        }
    } else {
        const TS *src = (const TS *)a.stage + row0 * B;
        TS *dst = (TS *)a.dGc;
        for (int lr = 0; lr < nrows; ++lr) {
            const int sl = sslot[lr / P];
            if (sl < 0)
                continue;
            for (int e = lane; e < B; e += 64)
                dst[((long)sl * P + lr % P) * B + e] = src[(long)lr * B + e];
        }
    }
}

// ---------------------------------------------------------------------------
// Fine-grained structure (section 3, Fig. 2(b)): a slice of P = Mx gate rows
// is its own region; it is cut into nb blocks of My batch columns (the last
// block narrower when My does not divide B) and the S = K blocks of lowest
// squared L2 norm are removed.  One wavefront owns one slice over every
// batch column (lane l holds columns l, l+64, ...): each My-lane group
// reduces its block's squares row by row with an xor butterfly (My/2, ...,
// 1) and folds the rows in order, so every lane ends with its block's score
// in a register.  A block is ranked against the others of its slice through
// scalar reads of their leader lanes; a ballot of the kept leaders gives the
// per-slice offset index.  The masked rows (removed blocks zeroed) go to dGc
// in the full [4H][B] layout; the bias gradient adds each masked row's sum.
// SRC selects where the gate-gradient values come from: computed from the
// cache (FS_CACHE), read from the staging matrix the element kernel wrote
// (FS_STAGE), or a given matrix (FS_GIVEN, selection only).
// ---------------------------------------------------------------------------
enum { FS_CACHE = 0, FS_STAGE = 1, FS_GIVEN = 2 };

__device__ __forceinline__ double readlane_f64(double v, int l) {
    const long long x = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane((int)(x & 0xffffffffLL), l);
    const int hi = __builtin_amdgcn_readlane((int)(x >> 32), l);
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

template <typename TS, int SRC, int MX>
__global__ __launch_bounds__(64) void cell_fine_kernel(CellArgs a) {
    constexpr int NJ = 4;  // 64-column chunks (B <= 256)
    const int lane = threadIdx.x;
    const int B = a.B, H = a.H, My = a.My, nb = a.nb, K = a.S;
    const long j = blockIdx.x;  // slice
    const long r0 = j * MX;
    const TS *__restrict__ gates = (const TS *)a.gates;
    const float *__restrict__ dHup = a.dH_up;
    const float *__restrict__ ct = a.c_t;
    const float *__restrict__ cp = a.c_prev;
    const float *__restrict__ dcin = a.dc_in;
    const TS *__restrict__ src = (const TS *)(SRC == FS_STAGE ? a.stage : a.dG_in);
    TS *dbg = (TS *)a.dbg;

    float vals[MX][NJ];
#pragma unroll
    for (int p = 0; p < MX; ++p) {
        const long r = r0 + p;
        const int g = (int)(r / H), u = (int)(r - (long)g * H);
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
            const int b = 64 * jj + lane;
            float val = 0.f;
            if (b < B) {
                if (SRC != FS_CACHE) {
                    val = st<TS>::load(src, r * B + b);
                } else {
                    const int e = u * B + b;
                    const float dh = sum_parts(dHup[e], a.dh_part + e, a.dh_nparts, a.dh_stride);
                    const float tc = tanhf(ct[e]);
                    const float o = st<TS>::load(gates, (long)(3 * H + u) * B + b);
                    if (g == 3) {
                        val = dh * tc * o * (1.f - o);
                    } else {
                        const float dcv = (dcin ? dcin[e] : 0.f) + dh * o * (1.f - tc * tc);
                        if (g == 1) {
                            const float f = st<TS>::load(gates, (long)(H + u) * B + b);
                            a.dc_out[e] = dcv * f;
                            val = dcv * cp[e] * f * (1.f - f);
                        } else {
                            const float i = st<TS>::load(gates, (long)u * B + b);
                            const float gg = st<TS>::load(gates, (long)(2 * H + u) * B + b);
                            val = g == 0 ? dcv * gg * i * (1.f - i) : dcv * i * (1.f - gg * gg);
                        }
                    }
                    val = st<TS>::rnd(val);
                    if (dbg)
                        st<TS>::store(dbg, r * B + b, val);
                }
            }
            vals[p][jj] = val;
        }
    }

    // block scores: per row a butterfly inside each My-lane group (columns
    // past B add zero), rows folded in increasing order
    double sc[NJ];
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) {
        sc[jj] = 0.0;
        if (64 * jj < B) {
#pragma unroll
            for (int p = 0; p < MX; ++p) {
                double q = (double)vals[p][jj] * (double)vals[p][jj];
                for (int off = My >> 1; off >= 1; off >>= 1)
                    q = q + shfl_xor_f64(q, off);
                sc[jj] = p == 0 ? q : sc[jj] + q;
            }
        }
    }
    const int bpc = 64 / My;  // blocks starting in one 64-column chunk
    const bool leader = (lane & (My - 1)) == 0;
    int cown[NJ];
    uint64_t kown[NJ];
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) {
        cown[jj] = jj * bpc + lane / My;
        kown[jj] = score_key(sc[jj]);
        if (a.scores && 64 * jj < B && leader && cown[jj] < nb)
            a.scores[j * nb + cown[jj]] = sc[jj];
    }
    // rank: a block is kept when fewer than nb - K blocks of its slice
    // outrank it (higher score, ties to the lower index, NaN highest)
    int beaten[NJ] = {};
#pragma unroll
    for (int j2 = 0; j2 < NJ; ++j2) {
        if (64 * j2 >= B)
            break;
        const int n2 = min(bpc, nb - j2 * bpc);
        for (int cb = 0; cb < n2; ++cb) {
            const int c2 = j2 * bpc + cb;
            const uint64_t k2 = score_key(readlane_f64(sc[j2], cb * My));
#pragma unroll
            for (int jj = 0; jj < NJ; ++jj)  // a block never outranks itself
                beaten[jj] += outranks_n(k2, c2, kown[jj], cown[jj]);
        }
    }
    bool keep[NJ];
    int base = 0;
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) {
        keep[jj] = beaten[jj] < nb - K;
        if (64 * jj < B) {
            const bool mine = leader && cown[jj] < nb && keep[jj];
            const uint64_t m = __ballot(mine);
            if (mine) {
                const int pos = base + __popcll(m & ((1ull << lane) - 1ull));
                a.idx[j * (nb - K) + pos] = cown[jj];
            }
            base += __popcll(m);
        }
    }

    // masked rows to dGc; bias gradient of the masked rows
    TS *dGc = (TS *)a.dGc;
#pragma unroll
    for (int p = 0; p < MX; ++p) {
        const long r = r0 + p;
        float rs = 0.f;
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
            const int b = 64 * jj + lane;
            if (b < B) {
                const float m = keep[jj] ? vals[p][jj] : 0.f;
                st<TS>::store(dGc, r * B + b, m);
                rs += m;
            }
        }
        if (SRC != FS_GIVEN && a.db) {
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1)
                rs += shfl_xor_f32(rs, off);
            if (lane == 0)
                a.db[r] += rs;
        }
    }
}

// db[r] (+)= the sum over steps t = t1 - 1 down to t0 (fp32, in that order)
// of row r's sum at step t (its chunk sums in chunk order) when the row's
// slice is kept at t (every step when idx is NULL).  Work-group x covers rows
// 64x .. 64x + 63, one per lane; its BG_WAVES wavefronts share out the steps
// of a pass of up to 64 (wavefront w: the pass's steps w, w + BG_WAVES, ...),
// so the loads of all of them are in flight together, and put each step's
// term in LDS (-0.0 when the slice was dropped, which adds nothing to any
// value); wavefront 0 then adds the pass's terms in decreasing step order.
// With EMAX / CMAX > 0 the kept-slice entries of the row's region (at most
// EMAX) and its chunk sums (at most CMAX) are read in unrolled loops.
constexpr int BG_WAVES = 8;

// Row r's term at step t of the bias gradient: its sum at step t (chunk sums
// in chunk order) when valid and its slice j is kept (every step when idx is
// NULL), else -0.0, which adds nothing to any value.  r and t must be in
// range also when not valid: the unrolled loops load unconditionally, from
// clamped positions, so that the loads of all steps are in flight together.
template <int EMAX, int CMAX, bool IDX>
__device__ __forceinline__ float bias_term(const float *chunk_rs, int nch, long G, long r, int t,
                                           bool valid, const int32_t *idx, int kept, long eb,
                                           int e1, long j) {
    const float *q = chunk_rs + ((long)t * G + r) * nch;
    float rs;
    if constexpr (CMAX > 0) {
        float qv[CMAX];
#pragma unroll
        for (int cc = 0; cc < CMAX; ++cc)
            qv[cc] = q[min(cc, nch - 1)];
        rs = qv[0];
#pragma unroll
        for (int cc = 1; cc < CMAX; ++cc)
            if (cc < nch)
                rs += qv[cc];
    } else {
        rs = q[0];
        for (int cc = 1; cc < nch; ++cc)
            rs += q[cc];
    }
    int hit = IDX ? 0 : 1;
    if constexpr (IDX) {  // e1 >= 1: the row's region has kept entries
        const int32_t *it = idx + (long)t * kept + eb;
        if constexpr (EMAX > 0) {
            int32_t iv[EMAX];
#pragma unroll
            for (int e = 0; e < EMAX; ++e)
                iv[e] = it[min(e, e1 - 1)];
#pragma unroll
            for (int e = 0; e < EMAX; ++e)
                hit |= (e < e1 && iv[e] == j) ? 1 : 0;
        } else {
            for (int e = 0; e < e1; ++e)
                hit |= it[e] == j ? 1 : 0;
        }
    }
    return (valid && hit) ? rs : -0.f;
}


template <int EMAX, int CMAX, bool IDX>
__global__ __launch_bounds__(64 * BG_WAVES) void bias_grad_kernel(float *db, const float *chunk_rs,
                                                                  int nch, long G, int t0, int t1,
                                                                  const int32_t *idx, int kept, int P,
                                                                  int R, int S, int accumulate) {
    constexpr int SPW = 64 / BG_WAVES;  // steps per wavefront and pass
    __shared__ float s_x[64][64];       // [step of the pass][row]
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const long r = blockIdx.x * 64L + lane;
    const bool in = r < G;
    const long rc = in ? r : G - 1;  // lanes past G read row G - 1's data
    const long j = rc / P;
    const int ks = R - S;
    const long eb = (j / R) * ks;
    const int e1 = (int)min((long)ks, kept - eb);
    float acc = (w == 0 && in && accumulate) ? db[r] : 0.f;
    for (int tb = t1 - 1; tb >= t0; tb -= 64) {
        float x[SPW];
#pragma unroll
        for (int k = 0; k < SPW; ++k) {
            const int t = tb - (w + BG_WAVES * k);
            const bool valid = t >= t0 && in;
            x[k] = bias_term<EMAX, CMAX, IDX>(chunk_rs, nch, G, rc, t >= t0 ? t : t0, valid, idx, kept,
                                         eb, e1, j);
        }
#pragma unroll
        for (int k = 0; k < SPW; ++k)
            s_x[w + BG_WAVES * k][lane] = x[k];
        __syncthreads();
        if (w == 0) {
            const int n = min(64, tb - t0 + 1);
            for (int i = 0; i < n; ++i)
                acc += s_x[i][lane];
        }
        __syncthreads();
    }
    if (w == 0 && in)
        db[r] = acc;
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
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
        out[i] = sum_parts(0.f, part + i, nparts, stride);
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

bool cell_split_ok(const CellArgs &a, int mode) {
    if ((long)a.H * a.B < 65536)
        return false;
    return mode == CELL_DENSE ||
           ((long)a.regions_per_wg * a.R <= 64 && (long)a.regions_per_wg * a.R * a.P <= 256);
}

template <typename TS>
static void launch_elem(const CellArgs &a, int mode, dim3 grid, hipStream_t s) {
    if (mode == CELL_SPARSE)
        hipLaunchKernelGGL((cell_elem_kernel<TS, CELL_SPARSE>), grid, dim3(EK_WAVES * 64), 0, s, a);
    else if (mode == CELL_GIVEN)
        hipLaunchKernelGGL((cell_elem_kernel<TS, CELL_GIVEN>), grid, dim3(EK_WAVES * 64), 0, s, a);
    else
        hipLaunchKernelGGL((cell_elem_kernel<TS, CELL_DENSE>), grid, dim3(EK_WAVES * 64), 0, s, a);
}

// CELL_GIVEN: the element kernel forms the chunk sums of squares of the given
// matrix (chunk_sq must be set), and the select kernel copies the kept rows
// from that matrix.
static hipError_t launch_cell_split(CellArgs a, int mode, bool bf16, hipStream_t s) {
    const int nch = (int)ceil_div(a.B, 64);
    dim3 ge((unsigned)ceil_div(a.H, EK_UNITS), (unsigned)nch);
    if (mode == CELL_GIVEN) {
        if (!a.chunk_sq || !a.dG_in)
            return hipErrorInvalidValue;
        a.stage = const_cast<void *>(a.dG_in);
    }
    if (bf16)
        launch_elem<bf16_t>(a, mode, ge, s);
    else
        launch_elem<float>(a, mode, ge, s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || mode == CELL_DENSE || (mode == CELL_SPARSE && a.defer_select))
        return e;
    const int grid = (int)ceil_div(a.nslices, (long)a.regions_per_wg * a.R);
    if (bf16)
        hipLaunchKernelGGL((cell_select_kernel2<bf16_t>), dim3(grid), dim3(64), 0, s, a);
    else
        hipLaunchKernelGGL((cell_select_kernel2<float>), dim3(grid), dim3(64), 0, s, a);
    return hipGetLastError();
}

// 32-row slices: four wavefronts per slice (eight rows each), so that the
// few slices (4H/32) still spread over the CUs.  Per-row block sums go to
// LDS; one thread per block folds the 32 rows in order, ranks and indexes.
template <typename TS, int SRC>
__global__ __launch_bounds__(256) void cell_fine32_kernel(CellArgs a) {
    constexpr int NJ = 4, RPW = 8;
    __shared__ double s_blk[32][64];
    __shared__ double s_sc[64];
    __shared__ int s_keep[64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int B = a.B, H = a.H, My = a.My, nb = a.nb, K = a.S;
    const long j = blockIdx.x;  // slice
    const long r0 = j * 32 + wave * RPW;
    const TS *__restrict__ gates = (const TS *)a.gates;
    const float *__restrict__ dHup = a.dH_up;
    const float *__restrict__ ct = a.c_t;
    const float *__restrict__ cp = a.c_prev;
    const float *__restrict__ dcin = a.dc_in;
    const TS *__restrict__ src = (const TS *)(SRC == FS_STAGE ? a.stage : a.dG_in);
    TS *dbg = (TS *)a.dbg;

    float vals[RPW][NJ];
#pragma unroll
    for (int p = 0; p < RPW; ++p) {
        const long r = r0 + p;
        const int g = (int)(r / H), u = (int)(r - (long)g * H);
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
            const int b = 64 * jj + lane;
            float val = 0.f;
            if (b < B) {
                if (SRC != FS_CACHE) {
                    val = st<TS>::load(src, r * B + b);
                } else {
                    const int e = u * B + b;
                    const float dh = sum_parts(dHup[e], a.dh_part + e, a.dh_nparts, a.dh_stride);
                    const float tc = tanhf(ct[e]);
                    const float o = st<TS>::load(gates, (long)(3 * H + u) * B + b);
                    if (g == 3) {
                        val = dh * tc * o * (1.f - o);
                    } else {
                        const float dcv = (dcin ? dcin[e] : 0.f) + dh * o * (1.f - tc * tc);
                        if (g == 1) {
                            const float f = st<TS>::load(gates, (long)(H + u) * B + b);
                            a.dc_out[e] = dcv * f;
                            val = dcv * cp[e] * f * (1.f - f);
                        } else {
                            const float i = st<TS>::load(gates, (long)u * B + b);
                            const float gg = st<TS>::load(gates, (long)(2 * H + u) * B + b);
                            val = g == 0 ? dcv * gg * i * (1.f - i) : dcv * i * (1.f - gg * gg);
                        }
                    }
                    val = st<TS>::rnd(val);
                    if (dbg)
                        st<TS>::store(dbg, r * B + b, val);
                }
            }
            vals[p][jj] = val;
        }
    }
    // this wavefront's rows' block sums (the My-lane butterfly's sum in each
    // block's first lane; columns past B add zero), all rows and chunks
    // interleaved
    {
        double q[RPW][NJ];
#pragma unroll
        for (int p = 0; p < RPW; ++p)
#pragma unroll
            for (int jj = 0; jj < NJ; ++jj)
                q[p][jj] = (double)vals[p][jj] * (double)vals[p][jj];
        auto sums = [&](auto w) {
            constexpr int W = decltype(w)::value;
#pragma unroll
            for (int p = 0; p < RPW; ++p)
#pragma unroll
                for (int jj = 0; jj < NJ; ++jj)
                    if (64 * jj < B)
                        q[p][jj] = lead_sum_f64<W>(q[p][jj]);
        };
        switch (My) {
        case 2: sums(std::integral_constant<int, 2>()); break;
        case 4: sums(std::integral_constant<int, 4>()); break;
        case 8: sums(std::integral_constant<int, 8>()); break;
        case 16: sums(std::integral_constant<int, 16>()); break;
        case 32: sums(std::integral_constant<int, 32>()); break;
        default: sums(std::integral_constant<int, 64>()); break;
        }
        const int lmy = __builtin_ctz(My);
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
            const int blk = (64 * jj + lane) >> lmy;
            if (64 * jj < B && (lane & (My - 1)) == 0 && blk < nb) {
#pragma unroll
                for (int p = 0; p < RPW; ++p)
                    s_blk[wave * RPW + p][blk] = q[p][jj];
            }
        }
    }
    __syncthreads();
    if (tid < nb) {  // score: the 32 rows folded in order
        double sc = s_blk[0][tid];
        for (int p = 1; p < 32; ++p)
            sc = sc + s_blk[p][tid];
        s_sc[tid] = sc;
        if (a.scores)
            a.scores[j * nb + tid] = sc;
    }
    __syncthreads();
    if (tid < nb) {  // kept when fewer than nb - K blocks outrank it
        const uint64_t kc = score_key(s_sc[tid]);
        int beaten = 0;
        for (int i = 0; i < nb; ++i)
            if (i != tid && outranks(score_key(s_sc[i]), i, kc, tid))
                ++beaten;
        s_keep[tid] = beaten < nb - K ? 1 : 0;
    }
    __syncthreads();
    if (tid < nb && s_keep[tid]) {
        int pos = 0;
        for (int i = 0; i < tid; ++i)
            pos += s_keep[i];
        a.idx[j * (nb - K) + pos] = tid;
    }
    TS *dGc = (TS *)a.dGc;
#pragma unroll
    for (int p = 0; p < RPW; ++p) {
        const long r = r0 + p;
        float rs = 0.f;
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
            const int b = 64 * jj + lane;
            if (b < B) {
                const float m = s_keep[b / My] ? vals[p][jj] : 0.f;
                st<TS>::store(dGc, r * B + b, m);
                rs += m;
            }
        }
        if (SRC != FS_GIVEN && a.db) {
            rs = lead_sum_f32<64>(rs);  // the 64-lane butterfly's sum in lane 0
            if (lane == 0)
                a.db[r] += rs;
        }
    }
}

// cell_fine4_kernel: 4-row slices with H % 4 == 0 at large shapes, the
// element kernel and the fine selection in one launch.  Work-group x covers
// units u0 = 4x .. 4x + 3 over all NCH = ceil(B / 64) batch chunks, one
// (unit, chunk) per wavefront (wavefront w: unit u0 + w % 4, chunk w / 4,
// lane l holding batch column 64 (w / 4) + l), as many loads in flight as the
// element kernel.  Rows g H + u0 .. g H + u0 + 3 are the whole slice
// (g H + u0) / 4, so the work-group holds four slices, one per gate.  Each
// wavefront forms its four gate values exactly as the element kernel does
// and puts each row's block sums (the butterfly inside My-lane groups) in
// LDS.  Wavefront g < 4 then scores the blocks of gate g's slice (the four
// rows folded in increasing order), ranks them by the total order
// cell_fine_kernel uses, with the comparisons shared out over all 64 lanes,
// and publishes a mask of the kept blocks.  Every wavefront stores its
// masked values; each row's masked values are summed per lane over the
// chunks in order, then over the 64 lanes, and added to db.  Values, scores,
// the order of every sum and the selection are those of the element kernel
// followed by cell_fine_kernel<TS, FS_STAGE, 4>.
template <typename TS, int NCH>
__global__ __launch_bounds__(256 * NCH) void cell_fine4_kernel(CellArgs a) {
    constexpr int NW = 4 * NCH;               // wavefronts
    constexpr int RPW = (16 + NW - 1) / NW;   // bias rows per wavefront (at most)
    __shared__ double s_q[4][4][64];          // [gate][row of the slice][block]
    __shared__ uint64_t s_keep[4];            // [gate]: kept blocks
    __shared__ double s_sc[4][64];            // [gate][block]: scores
    __shared__ float s_v[4][4][NCH][64];      // [gate][row][chunk][lane]: values
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int B = a.B, H = a.H, My = a.My, nb = a.nb, K = a.S;
    const int lmy = __builtin_ctz(My);  // My is a power of two
    const int p = w & 3, c = w >> 2;
    const int u0 = blockIdx.x * 4, u = u0 + p;  // H % 4 == 0: every unit is inside
    const int b = 64 * c + lane;
    const bool ok = b < B;
    float *db = a.db;

    float v[4];
    {
        const TS *__restrict__ gates = (const TS *)a.gates;
        const int e = u * B + (ok ? b : 0);
        float lg[4];
#pragma unroll
        for (int g = 0; g < 4; ++g)
            lg[g] = ok ? st<TS>::load(gates, (long)(g * H + u) * B + b) : 0.f;
        const float lct = ok ? a.c_t[e] : 0.f;
        const float lcp = ok ? a.c_prev[e] : 0.f;
        const float ldc = (ok && a.dc_in) ? a.dc_in[e] : 0.f;
        const float ldh =
            ok ? sum_parts<16>(a.dH_up[e], a.dh_part + e, a.dh_nparts, a.dh_stride) : 0.f;
        const float ig = lg[0], fg = lg[1], gg = lg[2], og = lg[3];
        const float tc = tanhf(lct);
        const float dcv = ldc + ldh * og * (1.f - tc * tc);
        v[0] = st<TS>::rnd(dcv * gg * ig * (1.f - ig));
        v[1] = st<TS>::rnd(dcv * lcp * fg * (1.f - fg));
        v[2] = st<TS>::rnd(dcv * ig * (1.f - gg * gg));
        v[3] = st<TS>::rnd(ldh * tc * og * (1.f - og));
        if (ok) {
            a.dc_out[u * B + b] = dcv * fg;
            TS *dbg = (TS *)a.dbg;
            if (dbg) {
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    st<TS>::store(dbg, (long)(g * H + u) * B + b, v[g]);
            }
        } else {
#pragma unroll
            for (int g = 0; g < 4; ++g)
                v[g] = 0.f;
        }
    }

    // db of the rows this wavefront finishes (row rr = 4 g + p of the
    // work-group), loaded now so that the loads complete during the selection
    float dbv[RPW];
#pragma unroll
    for (int k = 0; k < RPW; ++k) {
        const int rr = w + NW * k;
        dbv[k] = (db && rr < 16 && lane == 0) ? db[(long)(rr >> 2) * H + u0 + (rr & 3)] : 0.f;
    }

    // this row's block sums of squares in chunk c (columns past B add zero):
    // the My-lane butterfly of cell_fine_kernel, in each block's first lane
    {
        const int blk = c * (64 >> lmy) + (lane >> lmy);
        double q[4];
#pragma unroll
        for (int g = 0; g < 4; ++g)
            q[g] = (double)v[g] * (double)v[g];
        for (int off = My >> 1; off >= 16; off >>= 1) {
#pragma unroll
            for (int g = 0; g < 4; ++g)
                q[g] = q[g] + shfl_xor_f64(q[g], off);
        }
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            if (My >= 16)
                q[g] = q[g] + row_down_f64<8>(q[g]);
            if (My >= 8)
                q[g] = q[g] + row_down_f64<4>(q[g]);
            if (My >= 4)
                q[g] = q[g] + row_down_f64<2>(q[g]);
            q[g] = q[g] + row_down_f64<1>(q[g]);
        }
        if ((lane & (My - 1)) == 0 && blk < nb) {
#pragma unroll
            for (int g = 0; g < 4; ++g)
                s_q[g][p][blk] = q[g];
        }
    }
    if (db) {
#pragma unroll
        for (int g = 0; g < 4; ++g)
            s_v[g][p][c][lane] = v[g];
    }
    __syncthreads();

    if (w < 4) {  // wavefront g selects the blocks of gate g's slice
        // lane = q nbp + l (nbp: nb rounded up to a power of two) holds block
        // l and counts the blocks of the q-th share of the slice that
        // outrank it; the shares' counts are then added
        const int g = w;
        const long j = (long)g * (H / 4) + blockIdx.x;
        const int lnbp = nb > 1 ? 32 - __builtin_clz(nb - 1) : 0;  // nbp = 2^lnbp <= 64
        const int nbp = 1 << lnbp;
        const int l = lane & (nbp - 1), share = lane >> lnbp;
        const int len = (nb + (64 >> lnbp) - 1) >> (6 - lnbp);  // shares of 64 / nbp
        const bool own = l < nb;
        double sc = 0.0;
        if (own) {  // the four rows folded in increasing order
            sc = s_q[g][0][l];
#pragma unroll
            for (int r = 1; r < 4; ++r)
                sc = sc + s_q[g][r][l];
            if (share == 0) {
                s_sc[g][l] = sc;  // read back below by this wavefront only
                if (a.scores)
                    a.scores[j * nb + l] = sc;
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        const uint64_t kown = score_key(sc);
        int beaten = 0;  // a block never outranks itself
        const int c1 = min(nb, (share + 1) * len);
#pragma unroll 4
        for (int c2 = share * len; c2 < c1; ++c2)
            beaten += outranks_n(score_key(s_sc[g][c2]), c2, kown, l);
        if (nbp <= 16)
            beaten += (int)lane_xor_swap<16>((unsigned)beaten);
        if (nbp <= 32)
            beaten += (int)lane_xor_swap<32>((unsigned)beaten);
        for (int off = nbp; off < 16; off <<= 1)
            beaten += __shfl_xor(beaten, off, 64);
        // kept when fewer than nb - K blocks of the slice outrank it
        const bool mine = lane < nb && beaten < nb - K;  // lanes below nbp: share 0, l = lane
        const uint64_t m = __ballot(mine);
        if (mine)
            a.idx[j * (nb - K) + __popcll(m & ((1ull << lane) - 1ull))] = lane;
        if (lane == 0)
            s_keep[g] = m;
    }
    __syncthreads();

    // masked values to dGc
    TS *dGc = (TS *)a.dGc;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const float m = ((s_keep[g] >> (b >> lmy)) & 1ull) ? v[g] : 0.f;
        if (ok)
            st<TS>::store(dGc, (long)(g * H + u) * B + b, m);
    }
    if (!db)
        return;
    // bias gradient: the masked values per lane over the chunks in order,
    // then over the 64 lanes
    float rs[RPW];
#pragma unroll
    for (int k = 0; k < RPW; ++k) {
        const int rr = min(w + NW * k, 15);
        const uint64_t keep = s_keep[rr >> 2];
        rs[k] = 0.f;
#pragma unroll
        for (int jj = 0; jj < NCH; ++jj) {
            const int bj = 64 * jj + lane;
            if (bj < B)
                rs[k] += ((keep >> (bj >> lmy)) & 1ull) ? s_v[rr >> 2][rr & 3][jj][lane] : 0.f;
        }
    }
#pragma unroll
    for (int k = 0; k < RPW; ++k) {  // the 64-lane butterfly's sum in lane 0
        rs[k] = rs[k] + lane_xor_f32<32>(rs[k]);
        rs[k] = rs[k] + lane_xor_f32<16>(rs[k]);
        rs[k] = rs[k] + row_down_f32<8>(rs[k]);
        rs[k] = rs[k] + row_down_f32<4>(rs[k]);
        rs[k] = rs[k] + row_down_f32<2>(rs[k]);
        rs[k] = rs[k] + row_down_f32<1>(rs[k]);
    }
#pragma unroll
    for (int k = 0; k < RPW; ++k) {
        const int rr = w + NW * k;
        if (rr < 16 && lane == 0)
            db[(long)(rr >> 2) * H + u0 + (rr & 3)] = dbv[k] + rs[k];
    }
}

// cell_fine_sel_kernel: the selection of MX-row slices at large shapes
// from the element kernel's per-(row, block) sums (blk_sq, blk_rs), one
// wavefront per slice, lane b holding block b.  A block's score is its rows'
// sums of squares folded in increasing row order (the same values, in the
// same order, as cell_fine_kernel's and cell_fine32_kernel's); a block is
// kept when fewer than
// nb - K blocks of the slice outrank it.  The element kernel wrote the gate
// gradient to dGc; the removed blocks are zeroed there in place.  Each row's
// bias term is the sum of its kept blocks' sums by the 64-lane butterfly over
// the blocks (dropped ones add zero), added to db step by step.
template <typename TS, int MX>
__global__ __launch_bounds__(64) void cell_fine_sel_kernel(CellArgs a) {
    const int lane = threadIdx.x;
    const int B = a.B, My = a.My, nb = a.nb, K = a.S;
    const long j = blockIdx.x;  // slice
    const long r0 = j * MX;
    const bool own = lane < nb;
    const int bl = own ? lane : 0;  // lanes past the blocks read block 0
    double sq[MX];
    float rsv[MX];
#pragma unroll
    for (int p = 0; p < MX; ++p) {
        sq[p] = a.blk_sq[(r0 + p) * nb + bl];
        rsv[p] = a.blk_rs[(r0 + p) * nb + bl];
    }
    double sc = sq[0];
#pragma unroll
    for (int p = 1; p < MX; ++p)
        sc = sc + sq[p];
    if (!own)
        sc = 0.0;
    if (own && a.scores)
        a.scores[j * nb + lane] = sc;
    const uint64_t kown = score_key(sc);
    int beaten = 0;  // a block never outranks itself
    for (int c2 = 0; c2 < nb; ++c2)
        beaten += outranks_n(score_key(readlane_f64(sc, c2)), c2, kown, lane);
    const bool keep = own && beaten < nb - K;
    const uint64_t m = __ballot(keep);
    if (keep)
        a.idx[j * (nb - K) + __popcll(m & ((1ull << lane) - 1ull))] = lane;
    if (a.db) {
        float rs[MX];
#pragma unroll
        for (int p = 0; p < MX; ++p)
            rs[p] = lead_sum_f32<64>(keep ? rsv[p] : 0.f);
        if (lane == 0) {
#pragma unroll
            for (int p = 0; p < MX; ++p)
                a.db[r0 + p] += rs[p];
        }
    }
    // zero the removed blocks of the slice's rows
    TS *dGc = (TS *)a.dGc;
    const int lmy = __builtin_ctz(My);
    const int nch = (B + 63) / 64;
    for (int jj = 0; jj < nch; ++jj) {
        const int b = 64 * jj + lane;
        if (b < B && !((m >> (b >> lmy)) & 1ull)) {
#pragma unroll 8
            for (int p = 0; p < MX; ++p)
                st<TS>::store(dGc, (r0 + p) * B + b, 0.f);
        }
    }
}

template <typename TS, int SRC>
static void launch_fine_src(const CellArgs &a, hipStream_t s) {
    const dim3 grid((unsigned)(4L * a.H / a.P));
#define LSTMSS_FK(MX) hipLaunchKernelGGL((cell_fine_kernel<TS, SRC, MX>), grid, dim3(64), 0, s, a)
    switch (a.P) {
    case 1: LSTMSS_FK(1); break;
    case 2: LSTMSS_FK(2); break;
    case 4: LSTMSS_FK(4); break;
    case 8: LSTMSS_FK(8); break;
    case 16: LSTMSS_FK(16); break;
    default:
        hipLaunchKernelGGL((cell_fine32_kernel<TS, SRC>), grid, dim3(256), 0, s, a);
        break;
    }
#undef LSTMSS_FK
}

template <typename TS>
static hipError_t launch_fine_typed(const CellArgs &a, int mode, hipStream_t s) {
    if (mode == CELL_GIVEN) {
        launch_fine_src<TS, FS_GIVEN>(a, s);
    } else if (a.fine_fused && a.P == 4 && a.H % 4 == 0 && (long)a.H * a.B >= 65536) {
        const dim3 grid((unsigned)(a.H / 4));
        switch (ceil_div(a.B, 64)) {
        case 1: hipLaunchKernelGGL((cell_fine4_kernel<TS, 1>), grid, dim3(256), 0, s, a); break;
        case 2: hipLaunchKernelGGL((cell_fine4_kernel<TS, 2>), grid, dim3(512), 0, s, a); break;
        case 3: hipLaunchKernelGGL((cell_fine4_kernel<TS, 3>), grid, dim3(768), 0, s, a); break;
        default: hipLaunchKernelGGL((cell_fine4_kernel<TS, 4>), grid, dim3(1024), 0, s, a); break;
        }
    } else if (a.P != 4 && a.blk_sq && a.blk_rs && (long)a.H * a.B >= 65536) {
        // slices of 1, 2, 8, 16 or 32 rows at large shapes: the element
        // kernel writes the gate gradient and the per-block sums; the
        // selection reads only the sums (4-row slices take the fused kernel,
        // or the staging matrix and cell_fine_kernel)
        const int nch = (int)ceil_div(a.B, 64);
        dim3 ge((unsigned)ceil_div(a.H, EK_UNITS), (unsigned)nch);
        hipLaunchKernelGGL((cell_elem_kernel<TS, CELL_DENSE, true>), ge, dim3(EK_WAVES * 64), 0, s, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
        const dim3 gs((unsigned)(4L * a.H / a.P));
#define LSTMSS_FS(MX) hipLaunchKernelGGL((cell_fine_sel_kernel<TS, MX>), gs, dim3(64), 0, s, a)
        switch (a.P) {
        case 1: LSTMSS_FS(1); break;
        case 2: LSTMSS_FS(2); break;
        case 8: LSTMSS_FS(8); break;
        case 16: LSTMSS_FS(16); break;
        default: LSTMSS_FS(32); break;
        }
#undef LSTMSS_FS
    } else if (a.stage && (long)a.H * a.B >= 65536) {
        // large shapes: the element kernel forms each unit's four gate rows
        // once (one read of dh and the cache per unit), then the slices are
        // selected from its staging matrix.  It runs in its dense mode with
        // the staging matrix as output: the coarse chunk sums of squares are
        // not needed here
        const int nch = (int)ceil_div(a.B, 64);
        dim3 ge((unsigned)ceil_div(a.H, EK_UNITS), (unsigned)nch);
        CellArgs ea = a;
        ea.dGc = a.stage;
        hipLaunchKernelGGL((cell_elem_kernel<TS, CELL_DENSE>), ge, dim3(EK_WAVES * 64), 0, s, ea);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
        launch_fine_src<TS, FS_STAGE>(a, s);
    } else {
        launch_fine_src<TS, FS_CACHE>(a, s);
    }
    return hipGetLastError();
}

hipError_t launch_cell_fine(const CellArgs &a, int mode, bool bf16, hipStream_t s) {
    if ((a.P != 1 && a.P != 2 && a.P != 4 && a.P != 8 && a.P != 16 && a.P != 32) || a.My < 2 ||
        a.My > 64 ||
        (a.My & (a.My - 1)) != 0 || a.nb < 1 || a.nb > 64 || a.nb != (a.B + a.My - 1) / a.My ||
        a.B > 256 || a.S < 0 || a.S >= a.nb || (mode != CELL_SPARSE && mode != CELL_GIVEN) ||
        (4L * a.H) % a.P != 0)
        return hipErrorInvalidValue;
    return bf16 ? launch_fine_typed<bf16_t>(a, mode, s) : launch_fine_typed<float>(a, mode, s);
}

hipError_t launch_bias_grad(float *db, const float *chunk_rs, int nch, long G, int t0, int t1,
                            const int32_t *idx, int kept, int P, int R, int S, bool accumulate,
                            hipStream_t s) {
    const dim3 grid((unsigned)ceil_div(G, 64)), blk(64 * BG_WAVES);
    const bool unrolled = (!idx || R - S <= 8) && nch <= 4;
#define LSTMSS_BG(E, C, I)                                                                        \
    hipLaunchKernelGGL((bias_grad_kernel<E, C, I>), grid, blk, 0, s, db, chunk_rs, nch, G, t0, t1, \
                       idx, kept, P, R, S, accumulate ? 1 : 0)
    if (unrolled && idx)
        LSTMSS_BG(8, 4, true);
    else if (unrolled)
        LSTMSS_BG(8, 4, false);
    else if (idx)
        LSTMSS_BG(0, 0, true);
    else
        LSTMSS_BG(0, 0, false);
#undef LSTMSS_BG
    return hipGetLastError();
}

static bool cell_rows_ok(const CellArgs &a) {
    return (long)a.regions_per_wg * a.R * a.P <= 32 && (long)a.regions_per_wg * a.R <= 32 &&
           a.B <= 256;
}

template <typename TS, int M>
static void launch_rows(const CellArgs &a, int grid, hipStream_t s) {
    const int B = a.B;
#define LSTMSS_RK(L, J) hipLaunchKernelGGL((cell_rows_kernel<TS, M, L, J>), dim3(grid), dim3(RK_WAVES * 64), 0, s, a)
    if (B <= 1) LSTMSS_RK(1, 1);
    else if (B <= 2) LSTMSS_RK(2, 1);
    else if (B <= 4) LSTMSS_RK(4, 1);
    else if (B <= 8) LSTMSS_RK(8, 1);
    else if (B <= 16) LSTMSS_RK(16, 1);
    else if (B <= 32) LSTMSS_RK(32, 1);
    else if (B <= 64) LSTMSS_RK(64, 1);
    else if (B <= 128) LSTMSS_RK(64, 2);
    else if (B <= 192) LSTMSS_RK(64, 3);
    else LSTMSS_RK(64, 4);
#undef LSTMSS_RK
}

hipError_t launch_cell(const CellArgs &a, int mode, bool bf16, hipStream_t s) {
    // the split path of a given matrix needs the caller's chunk-sum scratch
    if (cell_split_ok(a, mode) && (mode != CELL_GIVEN || a.chunk_sq))
        return launch_cell_split(a, mode, bf16, s);
    if (cell_rows_ok(a)) {
        const int grid = (int)ceil_div(a.nslices, (long)a.regions_per_wg * a.R);
        if (bf16) {
            if (mode == CELL_DENSE) launch_rows<bf16_t, CELL_DENSE>(a, grid, s);
            else if (mode == CELL_SPARSE) launch_rows<bf16_t, CELL_SPARSE>(a, grid, s);
            else launch_rows<bf16_t, CELL_GIVEN>(a, grid, s);
        } else {
            if (mode == CELL_DENSE) launch_rows<float, CELL_DENSE>(a, grid, s);
            else if (mode == CELL_SPARSE) launch_rows<float, CELL_SPARSE>(a, grid, s);
            else launch_rows<float, CELL_GIVEN>(a, grid, s);
        }
        return hipGetLastError();
    }
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
