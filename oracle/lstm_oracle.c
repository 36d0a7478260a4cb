/*
 * CPU oracle for the structurally sparsified LSTM backward pass of
 * Zhu, Clemons, Pool, Rhu, Keckler, Xie, "Structurally Sparsified Backward
 * Propagation for Faster Long Short-Term Memory Training" (arXiv:1806.00512).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct
 * definition that the GPU library is checked against.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg may load it.  It shares
 * no code, header or table with the GPU library, and the GPU library never
 * calls it.
 *
 * Everything is plain fp64 loops in the order the method states them:
 *   - the LSTM cell (Hochreiter & Schmidhuber 1997, cited in the paper's
 *     introduction) with gate order i, f, g, o and no peepholes;
 *   - back-propagation through time, whose gate gradient (called dnet in the
 *     paper, section 3 and the Fig. 1 caption) feeds every weight and data
 *     gradient product;
 *   - coarse-grained structural sparsifying (section 3): dnet is cut into
 *     slices of P consecutive gate rows, R adjacent slices form a sparsifying
 *     region, and in each region the S slices with the smallest L2 norm are
 *     removed (S = R/2 gives 50 %, section 3 and Table 1);
 *   - the kept slices form a dense matrix plus an offset index array of the
 *     kept slices (section 3, the paragraph after Fig. 2); here the weight and
 *     data gradients are formed from the masked dense matrix, which is the
 *     plain definition of what the compacted products compute;
 *   - fine-grained structural sparsifying (section 3, Fig. 2(b); Table 1 for
 *     K): a slice of Mx rows is its own region, cut into blocks of My batch
 *     columns, and the K blocks of lowest L2 norm are removed from it.
 *
 * Readings where the paper is silent (each one is also listed in the design
 * notes of the repository):
 *   - a slice is P consecutive rows of the 4H x B gate-gradient matrix (rows
 *     in gate-major order [i; f; g; o]) spanning the whole batch;
 *   - the slice norm is compared squared (same ranking as the L2 norm);
 *   - ties keep the lower slice index; NaN ranks above +inf (kept);
 *   - a trailing partial region of r < R slices removes floor(S*r/R);
 *   - the cell-state recursion dc_{t-1} = dc * f uses the unsparsified dc;
 *   - the bias gradient sums the sparsified gate gradient;
 *   - a new mask is chosen at every time step;
 *   - fine: a trailing block narrower than My (when My does not divide B) is a
 *     block like the others, scored over its columns; K counts blocks.
 *
 * Score summation order (fixed so that a GPU selector fed the same fp32 gate
 * gradient bytes can be compared bit for bit):
 *   chunk c of a row holds the batch columns [64c, 64c + 64); its 64 squares
 *             (zero past B) are combined pairwise by index xor 32, 16, 8, 4,
 *             2, 1 (every position ends with the same value since fp64
 *             addition is commutative);
 *   rowsq(r) = ((chunk 0 + chunk 1) + chunk 2) + ... left fold over chunks;
 *   score(j) = (((rowsq(jP) + rowsq(jP+1)) + rowsq(jP+2)) + ...) left fold.
 * All of it in fp64; for fp32 inputs each square is exact in fp64, so whether
 * a compiler fuses multiply and add cannot change the result.
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared [-fopenmp].  The OpenMP
 * pragmas only split loops over independent output elements; each element is
 * always summed in the same order, so results do not depend on thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_ENOMEM (-3)

/* Number of threads the parallel loops use (1 without OpenMP). */
int oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Sets the number of threads of the parallel loops (n >= 1).  The loops only
 * split independent output elements among threads, so no result depends on
 * it; it serves timing on one core or all of them. */
void oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Round to the nearest bfloat16 value (8 significant bits, fp32 exponent
 * range, subnormal spacing 2^-133), ties to even.  Used only when the
 * storage type of a configuration is bf16. */
double oracle_round_bf16(double v)
{
    if (!isfinite(v) || v == 0.0)
        return v;
    double a = fabs(v);
    const double max_bf16 = ldexp(255.0, 120); /* 0x7F7F = (2 - 2^-7) * 2^127 */
    int e;
    frexp(a, &e); /* a = m * 2^e, m in [0.5, 1) */
    double spacing = (e - 1 >= -126) ? ldexp(1.0, e - 8) : ldexp(1.0, -133);
    double q = nearbyint(a / spacing) * spacing; /* default mode: ties to even */
    /* values that round beyond the largest finite bf16 go to infinity */
    if (q > max_bf16)
        q = INFINITY;
    return v < 0 ? -q : q;
}

static double sigmoid(double a) { return 1.0 / (1.0 + exp(-a)); }

/* ------------------------------------------------------------------------ */
/* Forward pass of one layer over T steps (support for the backward pass).   */
/*   x      [T][I][B]   layer input, batch contiguous                        */
/*   W      [4H][I+H]   [W_x | W_h], row blocks i, f, g, o                   */
/*   bias   [4H] or NULL                                                     */
/*   h0,c0  [H][B] or NULL (zero)                                            */
/* Outputs (the cache the backward pass reads):                              */
/*   gates  [T][4H][B]  activated i = s(a), f = s(a), g = tanh(a), o = s(a)  */
/*   c      [T+1][H][B] cell state, c[0] = c0                                */
/*   h      [T+1][H][B] hidden state, h[0] = h0                              */
/* bf16 != 0: the stored gates and h are rounded to bf16 (they are what the  */
/* bf16 configuration keeps); c, and the values c and h are computed from,   */
/* stay unrounded.                                                           */
/* ------------------------------------------------------------------------ */
int oracle_forward(int T, int B, int I, int H, const double *x, const double *W,
                   const double *bias, const double *h0, const double *c0, int bf16,
                   double *gates, double *c, double *h)
{
    if (T < 1 || B < 1 || I < 1 || H < 1 || !x || !W || !gates || !c || !h)
        return ORACLE_EINVAL;
    const long K = (long)I + H, G = 4L * H;
    double *a = (double *)malloc(sizeof(double) * G * B);
    if (!a)
        return ORACLE_ENOMEM;
    for (long e = 0; e < (long)H * B; ++e) {
        c[e] = c0 ? c0[e] : 0.0;
        double hv = h0 ? h0[e] : 0.0;
        h[e] = bf16 ? oracle_round_bf16(hv) : hv;
    }
    for (int t = 0; t < T; ++t) {
        const double *xt = x + (long)t * I * B;
        const double *hp = h + (long)t * H * B;
        /* pre-activations a = W [x_t; h_{t-1}] + bias */
#pragma omp parallel for schedule(static)
        for (long r = 0; r < G; ++r) {
            double *ar = a + r * B;
            for (int b = 0; b < B; ++b)
                ar[b] = bias ? bias[r] : 0.0;
            for (long k = 0; k < I; ++k) {
                double w = W[r * K + k];
                for (int b = 0; b < B; ++b)
                    ar[b] += w * xt[k * B + b];
            }
            for (long k = 0; k < H; ++k) {
                double w = W[r * K + I + k];
                for (int b = 0; b < B; ++b)
                    ar[b] += w * hp[k * B + b];
            }
        }
        double *gt = gates + (long)t * G * B;
        const double *cp = c + (long)t * H * B;
        double *cn = c + (long)(t + 1) * H * B;
        double *hn = h + (long)(t + 1) * H * B;
        for (long u = 0; u < H; ++u) {
            for (int b = 0; b < B; ++b) {
                double ig = sigmoid(a[(0 * H + u) * B + b]);
                double fg = sigmoid(a[(1 * H + u) * B + b]);
                double gg = tanh(a[(2 * H + u) * B + b]);
                double og = sigmoid(a[(3 * H + u) * B + b]);
                double cv = fg * cp[u * B + b] + ig * gg;
                double hv = og * tanh(cv);
                cn[u * B + b] = cv;
                hn[u * B + b] = bf16 ? oracle_round_bf16(hv) : hv;
                gt[(0 * H + u) * B + b] = bf16 ? oracle_round_bf16(ig) : ig;
                gt[(1 * H + u) * B + b] = bf16 ? oracle_round_bf16(fg) : fg;
                gt[(2 * H + u) * B + b] = bf16 ? oracle_round_bf16(gg) : gg;
                gt[(3 * H + u) * B + b] = bf16 ? oracle_round_bf16(og) : og;
            }
        }
    }
    free(a);
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Slice scores (section 3: the L2 norm of each slice, compared squared).     */
/* dG [rows][B]; rows must be a multiple of P; scores [rows / P].            */
/* ------------------------------------------------------------------------ */
static double chunk_sumsq(const double *row, int B, int c)
{
    double part[64], next[64];
    for (int l = 0; l < 64; ++l) {
        int b = 64 * c + l;
        part[l] = b < B ? row[b] * row[b] : 0.0;
    }
    for (int off = 32; off >= 1; off >>= 1) {
        for (int l = 0; l < 64; ++l)
            next[l] = part[l] + part[l ^ off];
        memcpy(part, next, sizeof(part));
    }
    return part[0];
}

static double row_sumsq(const double *row, int B)
{
    double s = chunk_sumsq(row, B, 0);
    for (int c = 1; 64 * c < B; ++c)
        s = s + chunk_sumsq(row, B, c);
    return s;
}

int oracle_scores(long rows, int B, int P, const double *dG, double *scores)
{
    if (rows < 1 || B < 1 || P < 1 || rows % P != 0 || !dG || !scores)
        return ORACLE_EINVAL;
    for (long j = 0; j < rows / P; ++j) {
        double s = row_sumsq(dG + (j * P) * B, B);
        for (int p = 1; p < P; ++p)
            s = s + row_sumsq(dG + (j * P + p) * B, B);
        scores[j] = s;
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Per-region selection (section 3; Table 1 for the (R, S) pairs).           */
/* Slices are grouped into consecutive regions of R.  In a full region the   */
/* S lowest-scored slices are removed; in a trailing region of r < R slices  */
/* floor(S*r/R) are removed.  Order used: higher score first, NaN highest,   */
/* equal scores -> lower slice index first.  keep[j] = 1 for kept slices.    */
/* ------------------------------------------------------------------------ */
static int outranks(double si, long i, double sj, long j)
{
    int ni = isnan(si), nj = isnan(sj);
    if (ni || nj) {
        if (ni && nj)
            return i < j;
        return ni; /* NaN outranks every number, +inf included */
    }
    if (si != sj)
        return si > sj;
    return i < j;
}

long oracle_removed_in_region(long r, int R, int S) { return (long)S * r / R; }

int oracle_select(long nslices, int R, int S, const double *scores, uint8_t *keep)
{
    if (nslices < 1 || R < 1 || R > 64 || S < 0 || S >= R || !scores || !keep)
        return ORACLE_EINVAL;
    for (long r0 = 0; r0 < nslices; r0 += R) {
        long r = nslices - r0 < R ? nslices - r0 : R;
        long nkeep = r - oracle_removed_in_region(r, R, S);
        for (long j = r0; j < r0 + r; ++j) {
            long beaten_by = 0;
            for (long i = r0; i < r0 + r; ++i)
                if (i != j && outranks(scores[i], i, scores[j], j))
                    ++beaten_by;
            keep[j] = beaten_by < nkeep ? 1 : 0;
        }
    }
    return ORACLE_OK;
}

/* Offset index array (section 3, after Fig. 2): the kept slice indices in   */
/* ascending order.  Returns how many were written.                         */
long oracle_kept_index(long nslices, const uint8_t *keep, int32_t *idx)
{
    long n = 0;
    for (long j = 0; j < nslices; ++j)
        if (keep[j])
            idx[n++] = (int32_t)j;
    return n;
}

/* Number of kept gate rows K' for a full 4H-row matrix. */
long oracle_kept_rows(long rows, int P, int R, int S)
{
    long nslices = rows / P, kept = 0;
    for (long r0 = 0; r0 < nslices; r0 += R) {
        long r = nslices - r0 < R ? nslices - r0 : R;
        kept += r - oracle_removed_in_region(r, R, S);
    }
    return kept * P;
}

/* ------------------------------------------------------------------------ */
/* Fine-grained structural sparsifying (section 3, Fig. 2(b); Table 1 for K; */
/* section 4 for M_y = 8, M_x = 4).  A slice is Mx consecutive gate rows over */
/* the whole batch and is its own sparsifying region; it is cut into blocks  */
/* of My consecutive batch columns (nb = ceil(B / My) of them, the last one   */
/* narrower when My does not divide B), and the K blocks of lowest L2 norm   */
/* (compared squared) are removed.  Sparsity = K / nb.                       */
/*                                                                          */
/* Block score order: for each of the Mx rows, the My squares of the block   */
/* (zero past B) combined pairwise by position xor My/2, ..., 2, 1; the rows */
/* then added in order.  scores [nslices][nb].                               */
/* ------------------------------------------------------------------------ */
static int is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

static double block_row_sumsq(const double *row, int B, int My, int cb)
{
    double part[64], next[64];
    for (int l = 0; l < My; ++l) {
        int b = cb * My + l;
        part[l] = b < B ? row[b] * row[b] : 0.0;
    }
    for (int off = My / 2; off >= 1; off >>= 1) {
        for (int l = 0; l < My; ++l)
            next[l] = part[l] + part[l ^ off];
        memcpy(part, next, sizeof(double) * My);
    }
    return part[0];
}

long oracle_fine_blocks(int B, int My) { return My > 0 ? (B + My - 1) / My : 0; }

int oracle_fine_scores(long rows, int B, int Mx, int My, const double *dG, double *scores)
{
    if (rows < 1 || B < 1 || Mx < 1 || rows % Mx != 0 || !is_pow2(My) || My > 64 || !dG ||
        !scores)
        return ORACLE_EINVAL;
    const long nb = oracle_fine_blocks(B, My);
    for (long s = 0; s < rows / Mx; ++s)
        for (long cb = 0; cb < nb; ++cb) {
            double v = block_row_sumsq(dG + (s * Mx) * B, B, My, (int)cb);
            for (int p = 1; p < Mx; ++p)
                v = v + block_row_sumsq(dG + (s * Mx + p) * B, B, My, (int)cb);
            scores[s * nb + cb] = v;
        }
    return ORACLE_OK;
}

/* keep [nslices][nb]: in every slice the K blocks ranked lowest are removed
 * (same order as the coarse selection: higher score first, NaN highest,
 * equal scores -> lower block index first). */
int oracle_fine_select(long nslices, long nb, int K, const double *scores, uint8_t *keep)
{
    if (nslices < 1 || nb < 1 || K < 0 || K >= nb || !scores || !keep)
        return ORACLE_EINVAL;
    for (long s = 0; s < nslices; ++s) {
        const double *sc = scores + s * nb;
        for (long j = 0; j < nb; ++j) {
            long beaten_by = 0;
            for (long i = 0; i < nb; ++i)
                if (i != j && outranks(sc[i], i, sc[j], j))
                    ++beaten_by;
            keep[s * nb + j] = beaten_by < nb - K ? 1 : 0;
        }
    }
    return ORACLE_OK;
}

/* Offset index array of the fine structure: per slice, the kept block
 * indices in ascending order, nb - K of them (-1 pads a forced mask that keeps
 * fewer).  bidx [nslices][nb - K]. */
void oracle_fine_kept_index(long nslices, long nb, int K, const uint8_t *keep, int32_t *bidx)
{
    for (long s = 0; s < nslices; ++s) {
        long n = 0;
        for (long j = 0; j < nb && n < nb - K; ++j)
            if (keep[s * nb + j])
                bidx[s * (nb - K) + n++] = (int32_t)j;
        while (n < nb - K)
            bidx[s * (nb - K) + n++] = -1;
    }
}

/* ------------------------------------------------------------------------ */
/* Backward pass through time of one layer, dense or structurally sparse.    */
/* Inputs are the forward cache (x, W, gates, c, h as oracle_forward made    */
/* them), the upstream gradient dH_up [T][H][B] of the loss with respect to  */
/* every h_t, and optional dhT / dcT [H][B] from later time (NULL = 0).      */
/* P, R, S: slice rows, slices per region, slices removed per region.        */
/*   S = 0 is the dense backward (every slice kept).                         */
/* forced_keep [T][4H/P] or NULL: use these masks instead of selecting.      */
/* Outputs: dX [T][I][B] (NULL skips), dW [4H][I+H], db [4H] (NULL skips),    */
/* dh0, dc0 [H][B] (NULL skips), keep_out [T][4H/P], idx_out [T][K'/P],       */
/* dG_out [T][4H][B] gate gradients before sparsifying (each NULL skips).    */
/* bf16 != 0: dG is rounded to bf16 before scoring, as that is the stored    */
/* operand the products consume.                                            */
/* ------------------------------------------------------------------------ */
/* fine != 0 selects the fine-grained structure: slices of P = Mx rows, blocks */
/* of My columns, K = S blocks removed per slice (R unused); forced_keep and  */
/* keep_out are then [T][4H/P][nb] and idx_out [T][4H/P][nb - S].           */
static int backward_impl(int T, int B, int I, int H, const double *x, const double *W,
                         const double *gates, const double *c, const double *h,
                         const double *dH_up, const double *dhT, const double *dcT, int fine,
                         int P, int R, int S, int My, int bf16, const uint8_t *forced_keep,
                         double *dX, double *dW, double *db, double *dh0, double *dc0,
                         uint8_t *keep_out, int32_t *idx_out, double *dG_out)
{
    const long K = (long)I + H, G = 4L * H, HB = (long)H * B;
    if (T < 1 || B < 1 || I < 1 || H < 1 || !x || !W || !gates || !c || !h || !dH_up || !dW)
        return ORACLE_EINVAL;
    if (P < 1 || G % P != 0)
        return ORACLE_EINVAL;
    if (!fine && (R < 1 || R > 64 || S < 0 || S >= R))
        return ORACLE_EINVAL;
    const long nb = fine ? oracle_fine_blocks(B, My) : 1;
    if (fine && (!is_pow2(My) || My > 64 || S < 0 || S >= nb))
        return ORACLE_EINVAL;
    const long nslices = G / P;
    const long nunits = fine ? nslices * nb : nslices;       /* mask entries per step */
    const long kept_slices = fine ? nslices * (nb - S) : oracle_kept_rows(G, P, R, S) / P;

    double *Wt = (double *)malloc(sizeof(double) * K * G);  /* W transposed */
    double *dG = (double *)malloc(sizeof(double) * G * B);
    double *dXH = (double *)malloc(sizeof(double) * K * B);
    double *dhrec = (double *)malloc(sizeof(double) * HB);
    double *dc = (double *)malloc(sizeof(double) * HB);
    double *scores = (double *)malloc(sizeof(double) * nunits);
    uint8_t *keep = (uint8_t *)malloc(nunits);
    int32_t *idx = (int32_t *)malloc(sizeof(int32_t) * nunits);
    if (!Wt || !dG || !dXH || !dhrec || !dc || !scores || !keep || !idx) {
        free(Wt); free(dG); free(dXH); free(dhrec); free(dc); free(scores); free(keep); free(idx);
        return ORACLE_ENOMEM;
    }
    for (long r = 0; r < G; ++r)
        for (long k = 0; k < K; ++k)
            Wt[k * G + r] = W[r * K + k];
    memset(dW, 0, sizeof(double) * G * K);
    if (db)
        memset(db, 0, sizeof(double) * G);
    for (long e = 0; e < HB; ++e) {
        dhrec[e] = dhT ? dhT[e] : 0.0;
        dc[e] = dcT ? dcT[e] : 0.0;
    }

    for (int t = T - 1; t >= 0; --t) {
        const double *gt = gates + (long)t * G * B;
        const double *ct = c + (long)(t + 1) * HB;   /* c_t     */
        const double *cp = c + (long)t * HB;         /* c_{t-1} */
        const double *xt = x + (long)t * I * B;      /* x_t     */
        const double *hp = h + (long)t * HB;         /* h_{t-1} */
        const double *dup = dH_up + (long)t * HB;

        /* Gate gradients (the data flow of Fig. 1). */
        for (long u = 0; u < H; ++u) {
            for (int b = 0; b < B; ++b) {
                long e = u * B + b;
                double ig = gt[(0 * H + u) * B + b], fg = gt[(1 * H + u) * B + b];
                double gg = gt[(2 * H + u) * B + b], og = gt[(3 * H + u) * B + b];
                double dh = dup[e] + dhrec[e];
                double tc = tanh(ct[e]);
                double dcv = dc[e] + dh * og * (1.0 - tc * tc);
                double d_o = dh * tc * og * (1.0 - og);
                double d_i = dcv * gg * ig * (1.0 - ig);
                double d_f = dcv * cp[e] * fg * (1.0 - fg);
                double d_g = dcv * ig * (1.0 - gg * gg);
                dG[(0 * H + u) * B + b] = d_i;
                dG[(1 * H + u) * B + b] = d_f;
                dG[(2 * H + u) * B + b] = d_g;
                dG[(3 * H + u) * B + b] = d_o;
                dc[e] = dcv * fg; /* dc_{t-1}: never sparsified */
            }
        }
        if (bf16)
            for (long e = 0; e < G * B; ++e)
                dG[e] = oracle_round_bf16(dG[e]);
        if (dG_out)
            memcpy(dG_out + (long)t * G * B, dG, sizeof(double) * G * B);

        /* Structural sparsifying: score, select (or take the forced mask). */
        if (forced_keep) {
            memcpy(keep, forced_keep + (long)t * nunits, nunits);
        } else if (fine) {
            oracle_fine_scores(G, B, P, My, dG, scores);
            oracle_fine_select(nslices, nb, S, scores, keep);
        } else {
            oracle_scores(G, B, P, dG, scores);
            oracle_select(nslices, R, S, scores, keep);
        }
        if (keep_out)
            memcpy(keep_out + (long)t * nunits, keep, nunits);
        if (idx_out) {
            if (fine) {
                oracle_fine_kept_index(nslices, nb, S, keep, idx_out + (long)t * kept_slices);
            } else {
                long n = oracle_kept_index(nslices, keep, idx);
                /* a forced mask may keep a different count; pad with -1 */
                for (long k = 0; k < kept_slices; ++k)
                    idx_out[(long)t * kept_slices + k] = k < n ? idx[k] : -1;
            }
        }
        /* Removed slices (coarse) or blocks (fine) contribute nothing to any
         * product. */
        if (fine) {
            for (long j = 0; j < nslices; ++j)
                for (long cb = 0; cb < nb; ++cb)
                    if (!keep[j * nb + cb])
                        for (long r = j * P; r < (j + 1) * P; ++r)
                            for (long b = cb * My; b < (cb + 1) * My && b < B; ++b)
                                dG[r * B + b] = 0.0;
        } else {
            for (long j = 0; j < nslices; ++j)
                if (!keep[j])
                    for (long e = j * P * B; e < (j + 1) * P * B; ++e)
                        dG[e] = 0.0;
        }

        /* Data gradients [dx_t; dh_{t-1}] = W^T dG. */
#pragma omp parallel for schedule(static)
        for (long k = 0; k < K; ++k) {
            double *out = dXH + k * B;
            for (int b = 0; b < B; ++b)
                out[b] = 0.0;
            for (long r = 0; r < G; ++r) {
                double w = Wt[k * G + r];
                for (int b = 0; b < B; ++b)
                    out[b] += w * dG[r * B + b];
            }
        }
        if (dX)
            memcpy(dX + (long)t * I * B, dXH, sizeof(double) * I * B);
        memcpy(dhrec, dXH + (long)I * B, sizeof(double) * HB);

        /* Weight gradients dW += dG [x_t; h_{t-1}]^T and db += dG 1. */
#pragma omp parallel for schedule(static)
        for (long r = 0; r < G; ++r) {
            const double *gr = dG + r * B;
            double *wr = dW + r * K;
            for (long k = 0; k < I; ++k) {
                double s = 0.0;
                for (int b = 0; b < B; ++b)
                    s += gr[b] * xt[k * B + b];
                wr[k] += s;
            }
            for (long k = 0; k < H; ++k) {
                double s = 0.0;
                for (int b = 0; b < B; ++b)
                    s += gr[b] * hp[k * B + b];
                wr[I + k] += s;
            }
            if (db) {
                double s = 0.0;
                for (int b = 0; b < B; ++b)
                    s += gr[b];
                db[r] += s;
            }
        }
    }
    if (dh0)
        memcpy(dh0, dhrec, sizeof(double) * HB);
    if (dc0)
        memcpy(dc0, dc, sizeof(double) * HB);
    free(Wt); free(dG); free(dXH); free(dhrec); free(dc); free(scores); free(keep); free(idx);
    return ORACLE_OK;
}

int oracle_backward(int T, int B, int I, int H, const double *x, const double *W,
                    const double *gates, const double *c, const double *h,
                    const double *dH_up, const double *dhT, const double *dcT, int P, int R,
                    int S, int bf16, const uint8_t *forced_keep, double *dX, double *dW,
                    double *db, double *dh0, double *dc0, uint8_t *keep_out, int32_t *idx_out,
                    double *dG_out)
{
    return backward_impl(T, B, I, H, x, W, gates, c, h, dH_up, dhT, dcT, 0, P, R, S, 0, bf16,
                         forced_keep, dX, dW, db, dh0, dc0, keep_out, idx_out, dG_out);
}

/* Fine-grained backward: slices of Mx rows, blocks of My columns, K blocks
 * removed per slice.  forced_keep / keep_out [T][4H/Mx][nb], idx_out
 * [T][4H/Mx][nb - K]. */
int oracle_backward_fine(int T, int B, int I, int H, const double *x, const double *W,
                         const double *gates, const double *c, const double *h,
                         const double *dH_up, const double *dhT, const double *dcT, int Mx,
                         int My, int K, int bf16, const uint8_t *forced_keep, double *dX,
                         double *dW, double *db, double *dh0, double *dc0, uint8_t *keep_out,
                         int32_t *idx_out, double *dG_out)
{
    return backward_impl(T, B, I, H, x, W, gates, c, h, dH_up, dhT, dcT, 1, Mx, 0, K, My, bf16,
                         forced_keep, dX, dW, db, dh0, dc0, keep_out, idx_out, dG_out);
}
