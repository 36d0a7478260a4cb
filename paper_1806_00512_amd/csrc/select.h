// Per-region selection of the coarse structure from per-row chunk sums of
// squares, shared by the select kernel and the data-gradient product's
// gathered-row prologue (section 3: in every region of R slices the S slices
// of lowest L2 norm are dropped, the kept ones take consecutive slots of the
// offset index).
#pragma once

#include "common.h"

namespace lstmss {

// True if slice i (score key ki) ranks above slice j (key kj) in a region:
// higher score, ties to the lower index (NaN keys rank highest).
__device__ __forceinline__ bool outranks(uint64_t ki, long i, uint64_t kj, long j) {
    return ki > kj || (ki == kj && i < j);
}

// outranks() as 0 / 1 without branches, for counting in unrolled loops
__device__ __forceinline__ int outranks_n(uint64_t ki, int i, uint64_t kj, int j) {
    return (int)((ki > kj) | ((ki == kj) & (i < j)));
}

struct SliceSel {
    double score;  // squared L2 norm of the lane's slice
    int slot;      // its slot in the step's offset index, -1 when dropped
    int pos;       // rank of the slot among the group's kept slices, -1 when dropped
    int nkept;     // kept slices of the whole group (the same in every lane)
};

// Score of slice j: the chunk sums of each of its P rows added in chunk
// order, then the rows in order (chunk_sq is [rows][nch], row r of slice j
// being j * P + p).
// The slice's P nch sums are contiguous; up to 16 of them are loaded at once
// (from clamped positions) and folded in the same order.
__device__ __forceinline__ double slice_score(const double *__restrict__ chunk_sq, int nch, long j,
                                              int P) {
    const int L = P * nch;
    const double *q = chunk_sq + j * L;
    if (L <= 16) {
        double v[16];
#pragma unroll
        for (int e = 0; e < 16; ++e)
            v[e] = q[min(e, L - 1)];
        double sc = 0.0, rs = 0.0;
        int end = nch - 1;  // last entry of the current row
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const bool in = e < L, start = e == end - nch + 1;
            rs = !in ? rs : start ? v[e] : rs + v[e];
            if (in && e == end) {  // row e / nch complete
                sc = e == nch - 1 ? rs : sc + rs;
                end += nch;
            }
        }
        return sc;
    }
    double sc = 0.0;
    for (int p = 0; p < P; ++p) {
        const double *qr = q + p * nch;
        double rs = qr[0];
        for (int c = 1; c < nch; ++c)
            rs = rs + qr[c];
        sc = p == 0 ? rs : sc + rs;
    }
    return sc;
}

// One wavefront: lane j ranks and places slice j0 + j (score sc) of the
// group [j0, j0 + nsl) (j0 a multiple of R, nsl <= 64, whole regions except
// a trailing partial one at the end of the slice list); a region of r slices
// keeps r - floor(S r / R); the kept slices of region q take slots
// q (R - S), q (R - S) + 1, ... in ascending slice order.  Lanes >= nsl
// return slot -1.
__device__ __forceinline__ SliceSel rank_slices(double sc, long j0, int nsl, int R, int S,
                                                long nslices) {
    const int lane = threadIdx.x & 63;
    const int j = lane;
    const bool valid = j < nsl;
    if (!valid)
        sc = 0.0;
    const uint64_t kj = score_key(sc);
    const long gj = j0 + j;
    // regions start at multiples of R and j0 is one, so a region's slices
    // are the lanes [ls, ls + rlen) of this wavefront
    const int ls = valid ? (int)((gj / R) * R - j0) : 0;
    const int rlen = valid ? (int)min((long)R, nslices - (j0 + ls)) : 0;
    const int nkeep = rlen - (S * rlen) / R;
    int beaten = 0;  // a slice never outranks itself
#pragma unroll 8
    for (int i = 0; i < R; ++i) {
        const int src = (ls + i) & 63;
        const uint64_t ki = (uint64_t)__shfl((long long)kj, src, 64);
        beaten += i < rlen ? outranks_n(ki, src, kj, j) : 0;
    }
    const bool keep = valid && beaten < nkeep;
    const uint64_t ball = __ballot(keep);
    const uint64_t lower = j ? (~0ull >> (64 - j)) : 0ull;
    const uint64_t below = lower & ~(ls ? (~0ull >> (64 - ls)) : 0ull);
    SliceSel r;
    r.score = sc;
    r.slot = keep ? (int)((gj / R) * (R - S) + __popcll(ball & below)) : -1;
    r.pos = keep ? __popcll(ball & lower) : -1;
    r.nkept = __popcll(ball);
    return r;
}

// Scores (from the chunk sums), ranks and places the group's slices.
__device__ __forceinline__ SliceSel select_slices(const double *__restrict__ chunk_sq, int nch,
                                                  long j0, int nsl, int P, int R, int S,
                                                  long nslices) {
    const int j = threadIdx.x & 63;
    const double sc = j < nsl ? slice_score(chunk_sq, nch, j0 + j, P) : 0.0;
    return rank_slices(sc, j0, nsl, R, S, nslices);
}

} // namespace lstmss
