// Kernel parameter blocks and launchers (internal to liblstmss).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/lstmss.h"

namespace lstmss {

enum CellMode { CELL_DENSE = 0, CELL_SPARSE = 1, CELL_GIVEN = 2 };

// One backward time step of the elementwise gate-gradient work, fused with
// slice scoring, per-region selection and compaction of the kept rows.
struct CellArgs {
    int B, H, I;
    int P, R, S;
    long nslices;          // 4H / P
    int regions_per_wg;    // work-group tile in regions
    // inputs of step t (storage type is the kernel's template type)
    const void *gates;     // [4H][B] activated i, f, g, o
    const float *c_t;      // [H][B]
    const float *c_prev;   // [H][B]
    const float *dH_up;    // [H][B]
    const float *dh_part;  // dh_rec as dh_nparts partial sums spaced dh_stride, or NULL
    int dh_nparts;
    long dh_stride;
    const float *dc_in;    // [H][B] or NULL (zero)
    float *dc_out;         // [H][B]
    const void *dG_in;     // CELL_GIVEN only: [4H][B]
    // outputs
    void *dGc;             // [K'][B]
    int32_t *idx;          // [K'/P] (sparse modes)
    float *db;             // [4H] accumulated over kept rows, or NULL
    void *dbg;             // [4H][B] or NULL
    double *scores;        // [4H/P] or NULL
    int defer_select;      // split path: element kernel only, the dh product selects
    // split variant (large shapes): staging matrix and per-(row, chunk) sums
    void *stage;           // [4H][B] gate gradient before selection (sparse)
    double *chunk_sq;      // [4H][ceil(B/64)] fp64 chunk sums of squares
    float *chunk_rs;       // [4H][ceil(B/64)] fp32 chunk row sums
    // fine-grained structure: slices of P rows cut into nb blocks of My batch
    // columns, S blocks removed per slice; dGc is then the masked [4H][B]
    // matrix, idx [4H/P][nb - S] the kept blocks and scores [4H/P][nb]
    int My, nb;
    int fine_fused;        // 4-row slices, H % 4 == 0, large shapes: one fused kernel
    // 32-row slices at large shapes: per (row, block) sums of squares and
    // sums of one step, [4H][nb], written by the element kernel
    double *blk_sq;
    float *blk_rs;
};

// Data gradient [dx_t; dh_{t-1}] = W_c^T dG_c, split over K into partials.
// One launch covers `steps` consecutive time steps (grid z = step * splitk +
// split); step s reads Gc + s*gc_step, idx + s*idx_step and writes
// part + s*out_step + split*part_stride.
struct Gemm1Args {
    const void *W;         // [4H][ldw]
    long ldw;              // I + H
    const void *Gc;        // [Kp][N] of the first step
    const int32_t *idx;    // [Kp/P] kept slices of the first step, or NULL (identity)
    int P;
    long Kp;
    int M, m_begin, N;     // output rows [m_begin, M), columns N = B
    int out_row0;          // output row m is stored at row m - out_row0
    int m_lo;              // tile origin (m_begin rounded down for aligned loads; set by the launcher)
    float *part;           // [splitk][rows][N] per step
    long part_stride;      // rows * N
    int splitk;
    long k_chunk;
    int steps;
    long gc_step, idx_step, out_step;
    int tm, tn;            // tile rows / columns, 0 = chosen by the launcher
    int kcol0;             // launch_gemm_fwd only: first W column of the product
    int waves;             // wavefronts per work-group: 0 or 4, or 8 for 128-row tiles
    // fine structure with 32-row slices and 32-column blocks (Gc the masked
    // matrix, no gather): kept block indices of the first step,
    // [4H/32][fkept], fidx_step entries per step; MFMAs of removed blocks
    // are skipped.  NULL otherwise.
    const int32_t *fidx;
    int fkept;
    long fidx_step;
    int dma;               // 1: fp32 stages go global -> LDS directly where the shape allows
                           // (same bits as the register-staged loads of 0)
    // coarse selection inside the product (one step, DMA stages, idx NULL):
    // Gc is then the staging matrix [4H][N] of the step; the product ranks
    // the slices of its splits' regions from sel_sq, gathers both operands
    // through the kept rows and writes the compacted matrix sel_gc
    // [Kp][N] and the offset index sel_idx [kept].  NULL otherwise.
    const double *sel_sq;  // [4H][sel_nch] chunk sums of squares
    int sel_nch, sel_R, sel_S;
    long sel_nslices;
    void *sel_gc;
    int32_t *sel_idx;
};

// Weight gradient dW[rows] += dG_c [x_t; h_{t-1}]^T (rows scattered by idx).
struct Gemm2Args {
    const void *Gc;        // [Kp][B]
    const int32_t *idx;    // [Kp/P] or NULL
    int P;
    long Kp;
    const void *xt;        // [I][B]
    const void *hp;        // [H][B]
    int I, H, B;
    float *dW;             // [4H][I+H]
};

// Weight gradient of the whole sequence in one launch:
//   dW = sum_t dG_t [x_t; h_{t-1}]^T   (dense: every row; sparse: the kept
//   rows of each step are accumulated into their original rows).
struct WgradArgs {
    const void *Gc;        // [T][Kp][B] compacted gate gradients of every step
    const int32_t *idx;    // [T][kept] kept slice indices (sparse) or NULL
    const void *x;         // [T][I][B]
    const void *h;         // [T+1][H][B] (step t reads h[t] = h_{t-1})
    int T, I, H, B;
    int Kp, kept;          // kept rows / kept slices per step
    int P, R, S;
    int greg;              // regions per work-group group (sparse)
    int BC;                // batch columns staged per iteration
    int t_begin, t_end;    // time steps [t_begin, t_end) of this launch
    int accumulate;        // 0: dW = sum; 1: dW += sum, continuing from the stored dW
    float *dW;             // [4H][I+H]
    // fine structure with 32-row slices and 32-column blocks (dense layout,
    // Gc the masked matrix): kept block indices [T][4H/32][fkept]; a row
    // group skips the batch chunks of its removed blocks.  NULL otherwise.
    const int32_t *fidx;
    int fkept;
    int fskip;             // 1: skip removed blocks; 0: multiply them (same bits)
    int dma;               // 1: chunks go global -> LDS directly where the shape allows
                           // (same bits as the register-staged loads of 0)
    int big;               // bf16 with DMA chunks: 1 takes the 256 x 256-tile kernel
                           // where it applies (its own summation order)
};

// Forward cell update from the pre-activation pieces of one step.
struct FwdActArgs {
    const float *zx;       // [4H][B] input projection W_x x_t
    const float *part;     // [nparts][4H][B] recurrent partials W_h h_{t-1}
    int nparts;
    long part_stride;      // 4H * B
    const float *bias;     // [4H] or NULL
    const float *cp;       // [H][B] c_{t-1}
    int H, B;
    void *gates;           // [4H][B] activated gates (storage type)
    float *cn;             // [H][B] c_t
    void *hn;              // [H][B] h_t (storage type)
    void *hout;            // [H][B] or NULL
};

// One forward step: a = W [x_t; h_{t-1}] + b, activations, cell update.
struct FwdArgs {
    const void *W;
    const float *bias;     // [4H] or NULL
    const void *xt;        // [I][B]
    const void *hp;        // [H][B]
    const float *cp;       // [H][B]
    int I, H, B;
    void *gates;           // [4H][B]
    float *cn;             // [H][B]
    void *hn;              // [H][B]
    void *hout;            // [H][B] or NULL
};

hipError_t launch_cell(const CellArgs &a, int mode, bool bf16, hipStream_t s);
// Fine-grained structure (mode CELL_SPARSE or CELL_GIVEN): P in {1,2,4,8,16,32},
// My a power of two in [2, 64], nb = ceil(B/My) <= 64, B <= 256.  With
// stage set and H*B >= 65536, CELL_SPARSE runs the element kernel into stage
// (and chunk_sq, chunk_rs) before the selection; db (when set) accumulates
// the masked row sums.
hipError_t launch_cell_fine(const CellArgs &a, int mode, bool bf16, hipStream_t s);
size_t cell_lds_bytes(const CellArgs &a, int mode);
// True when launch_cell uses the split (element kernel + select kernel) path;
// the bias gradient then comes from chunk_rs through launch_bias_grad.
bool cell_split_ok(const CellArgs &a, int mode);
hipError_t launch_bias_grad(float *db, const float *chunk_rs, int nch, long G, int t0, int t1,
                            const int32_t *idx, int kept, int P, int R, int S, bool accumulate,
                            hipStream_t s);
hipError_t launch_gemm1(Gemm1Args a, bool bf16, hipStream_t s);
// True when launch_gemm1 accepts a (selection inside the product, sel_sq set).
bool gemm1_select_ok(Gemm1Args a, bool bf16);
hipError_t launch_gemm2(const Gemm2Args &a, bool bf16, hipStream_t s);
// Forward products part[z][m][n] = sum over k in split z of
// W[m][kcol0 + k] G[k][n] (rows m in [0, M), contraction length Kp).
hipError_t launch_gemm_fwd(Gemm1Args a, bool bf16, hipStream_t s);
hipError_t launch_fwd_act(const FwdActArgs &a, bool bf16, hipStream_t s);
// Training step: W -= lr dW (storage type), b -= lr db; and the regression
// loss gradient dH = (h - y) / B with per-block loss partials (nparts <= 1024
// blocks, their sum written to parts[nparts]).
hipError_t launch_sgd(void *W, const float *dW, long nw, float *b, const float *db, long nb,
                      float lr, bool bf16, hipStream_t s);
hipError_t launch_mse(const void *h, const float *y, float *dH, long n, float inv_b,
                      double *parts, int nparts, bool bf16, hipStream_t s);
// Bidirectional layer edges (time reversal of the reverse direction):
// dst[s] = src[T-1-s] over steps of `words` 4-byte words; out[t] =
// [hf[t]; hr[T-1-t]] ([T][2H][B]); df[t] = dH[t][:H], dr[T-1-t] = dH[t][H:];
// out[t] = a[t] + b[T-1-t] ([T][I][B]).
hipError_t launch_reverse(const void *src, void *dst, int T, long words, hipStream_t s);
hipError_t launch_bidir_join(const void *hf, const void *hr, void *out, int T, long HB, bool bf16,
                             hipStream_t s);
hipError_t launch_bidir_split(const float *dH, float *df, float *dr, int T, long HB, hipStream_t s);
hipError_t launch_sum_rev(const float *a, const float *b, float *out, int T, long IB,
                          hipStream_t s);
// Returns hipErrorNotSupported when the structure needs more routing tiles
// than the batched kernel holds (the caller then uses launch_gemm2 per step).
hipError_t launch_wgrad(WgradArgs a, bool sparse, bool bf16, hipStream_t s);
bool wgrad_supported(int P, int R, int S);
hipError_t launch_fwd_step(const FwdArgs &a, bool bf16, hipStream_t s);
hipError_t launch_fill(float *p, long n, float v, hipStream_t s);
hipError_t launch_copy_in(float *dst, const float *src, long n, hipStream_t s); // src NULL -> zero
hipError_t launch_reduce_parts(float *out, const float *part, int nparts, long stride, long n,
                               hipStream_t s);
hipError_t launch_h0_store(void *dst, const float *src, long n, bool bf16, hipStream_t s);

// Host-side pieces of the C ABI shared with the entry point that allocates
// nothing (noalloc.hip): the last-error setter, the standalone selection's
// scratch size and the selection itself (hooks: timing hooks enabled).
int32_t set_error(int32_t code, const char *msg);
int64_t select_scratch_bytes(const lstmss_dims *d, float sparsity, const lstmss_structure *s);
int32_t select_compact_impl(const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                            const void *dG, void *dG_c, int32_t *idx, double *scores, void *ws,
                            size_t ws_bytes, void *stream, bool hooks);

// Tile constants shared by the host-side sizing code.
constexpr int GEMM1_TK = 64;       // granularity of a split's k range
constexpr int GEMM1_KC_MAX = 2048; // gathered rows looked up into LDS at a time
// fine structure fast path: at most this many 32-row slices per product (4H <= 16384)
constexpr int FINE_MAX_SLICES = 512;
void gemm1_tile(bool bf16, int N, long rows, long zdim, int *tm, int *tn);
int gemm1_wgs_per_cu(int tm, int tn);

} // namespace lstmss
