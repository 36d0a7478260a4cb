/*
 * lstmss — structurally sparsified LSTM backward pass on AMD Instinct MI355X
 * (gfx950).  C ABI of liblstmss.so.
 *
 * Method: Zhu, Clemons, Pool, Rhu, Keckler, Xie, "Structurally Sparsified
 * Backward Propagation for Faster Long Short-Term Memory Training",
 * arXiv:1806.00512.  In the backward pass of an LSTM layer the gate gradient
 * dnet (4H x B per time step) is cut into slices of P consecutive gate rows,
 * R adjacent slices form a sparsifying region, and in every region the S
 * slices with the smallest L2 norm are dropped (section 3; S/R is the
 * sparsity, Table 1).  The kept slices form a dense matrix plus an offset
 * index array (section 3, after Fig. 2), and the weight and data gradient
 * products run on that compacted matrix (section 4, custom operation).
 *
 * Conventions for every entry point
 *   - Tensor pointers are DEVICE pointers owned by the caller.  The library
 *     never allocates device memory; scratch comes from the caller's
 *     workspace `ws` of `ws_bytes` bytes (query the size first).
 *   - Row-major, batch B is the contiguous (last) dimension everywhere.
 *   - W = [W_x | W_h] is 4H x (I+H); its row blocks are the gates in the order
 *     i, f, g, o (rows [0,H) = i, [H,2H) = f, [2H,3H) = g, [3H,4H) = o).
 *   - `dtype` is the storage type of x, W, h_out and the cache's gates and h
 *     (fp32 or bf16).  Accumulation is fp32.  Biases, h0, c0, every gradient
 *     (dH_up, dX, dW, db, dh0, dc0) and the cell state are fp32.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream)
 *     and the calls return without synchronising the host.
 *   - Calls return LSTMSS_OK (0) or a negative error code; nothing is
 *     enqueued when an argument check fails.  lstmss_last_error() gives the
 *     calling thread's detail message for the last failure.
 *   - Calls that overlap in time on different streams must use different
 *     workspaces and outputs.
 */
#ifndef LSTMSS_H
#define LSTMSS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LSTMSS_VERSION 1

typedef enum { LSTMSS_F32 = 0, LSTMSS_BF16 = 1 } lstmss_dtype;

/* Sparsifying structure kinds (section 3, Fig. 2): COARSE drops whole
 * P-row slices inside regions of R slices; FINE drops My-column blocks of
 * Mx-row slices, each slice being its own region. */
typedef enum { LSTMSS_COARSE = 0, LSTMSS_FINE = 1 } lstmss_kind;

enum {
    LSTMSS_OK = 0,
    LSTMSS_ERR_INVALID_ARG = -1, /* null required pointer, bad size or structure */
    LSTMSS_ERR_UNSUPPORTED = -2, /* valid but not built (a size past a kernel limit) */
    LSTMSS_ERR_WORKSPACE = -3,   /* ws_bytes smaller than the size query returned */
    LSTMSS_ERR_HIP = -4          /* a HIP runtime call failed (see lstmss_last_error) */
};

/* One layer over the whole sequence: T steps, batch B, input size I,
 * hidden size H, storage dtype (lstmss_dtype). */
typedef struct {
    int32_t T, B, I, H;
    int32_t dtype;
} lstmss_dims;

/* COARSE: P gate rows per slice, R slices per region (1 <= R <= 64).
 * The number of slices removed per region is S = sparsity * R, which must be
 * an integer (within 1e-6) with 0 <= S < R.  4H must be a multiple of P.
 * When 4H/P is not a multiple of R, the last region has r < R slices and
 * removes floor(S*r/R).  My, Mx are ignored.
 * FINE: a slice is Mx consecutive gate rows (Mx in 1..32 dividing 32 and
 * 4H) over the whole batch, cut into nb = ceil(B/My) blocks of My batch
 * columns (My a power of two in 2..64; the last block is narrower when My
 * does not divide B; nb <= 64, B <= 256).  In every slice the K = sparsity *
 * nb blocks of smallest L2 norm are zeroed (K an integer within 1e-6,
 * 0 <= K < nb).  P, R are ignored.  With Mx = My = 32 (blocks shaped like
 * the 32 x 32 MFMA operand blocks), fp32 storage, B a multiple of 32 and
 * 4H <= 16384, the gradient products skip the removed blocks'
 * multiplications (same results bit for bit); other block shapes, and bf16
 * storage (whose products are bound by their loads, not their
 * multiplications), run the products on the masked matrix. */
typedef struct {
    int32_t kind;
    int32_t P, R;
    int32_t My, Mx;
} lstmss_structure;

int32_t lstmss_version(void);
const char *lstmss_strerror(int32_t code);
/* Detail of the calling thread's last failed call ("" if none). */
const char *lstmss_last_error(void);

/* Bytes of the forward cache written by lstm_fwd_cache and read by the
 * backward calls: activated gates [T][4H][B] (dtype), cell state
 * [T+1][H][B] (fp32) and hidden state [T+1][H][B] (dtype).  <0 on error. */
int64_t lstmss_cache_bytes(const lstmss_dims *d);

/* Rows of the per-step gate-gradient matrix the products run on: for
 * COARSE K' = P x (number of kept slices per step), 4H when sparsity is 0;
 * for FINE always 4H (removed blocks are zero in place).  <0 on error. */
int64_t lstmss_kept_rows(const lstmss_dims *d, float sparsity, const lstmss_structure *s);

/* How lstm_bwd_structsparse runs the gate path of a call with these
 * arguments under the current options, for a 256-byte aligned weight matrix
 * and workspace: *flags gets LSTMSS_INFO_SPLIT_GATES when the gate gradient
 * and the selection of section 3 are computed by an element kernel and a
 * selection step (H * B >= 65536), and LSTMSS_INFO_SELECT_IN_PRODUCT when
 * that selection and the compaction run inside the per-step dh product
 * (LSTMSS_OPT_GEMM_SELECT) instead of a kernel of their own.  Results are
 * the same bits either way; this is for profiling and accounting.  0 or a
 * negative error code (no GPU work). */
enum { LSTMSS_INFO_SPLIT_GATES = 1, LSTMSS_INFO_SELECT_IN_PRODUCT = 2 };
int32_t lstmss_bwd_info(const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                        int32_t *flags);

/* Entries of the per-step index written by the selection: COARSE K'/P kept
 * slice indices; FINE (4H/Mx) x (nb - K) kept block indices.  <0 on error. */
int64_t lstmss_index_entries(const lstmss_dims *d, float sparsity, const lstmss_structure *s);

/* Workspace bytes needed by lstm_bwd_structsparse with these arguments
 * (sparsity 0 gives a size that serves both lstm_bwd_dense and
 * lstm_bwd_structsparse at sparsity 0).  <0 on error. */
int64_t lstmss_workspace_bytes(const lstmss_dims *d, float sparsity, const lstmss_structure *s);

/* Workspace bytes for lstm_fwd_cache's batched path: the fp32 input
 * projection of every step plus one step's recurrent split-K partials.
 * <0 on error. */
int64_t lstmss_fwd_workspace_bytes(const lstmss_dims *d);

/* Forward pass of one LSTM layer, keeping what the backward pass reads
 * (the paper's forward computes the gate activations, section 4).
 *   a_t = W [x_t; h_{t-1}] + b;  i, f, o = sigmoid, g = tanh of a_t's blocks;
 *   c_t = f*c_{t-1} + i*g;  h_t = o*tanh(c_t).
 *   x      [T][I][B] dtype            W [4H][I+H] dtype
 *   b      [4H] fp32, NULL = 0        h0, c0 [H][B] fp32, NULL = 0
 *   h_out  [T][H][B] dtype (h_1..h_T), may be NULL
 *   cache  lstmss_cache_bytes(d) bytes, written
 *   ws     lstmss_fwd_workspace_bytes(d) bytes: the input projection W_x x_t
 *          of all steps runs as one product, then every step runs its
 *          recurrent product W_h h_{t-1} split over k and a cell-update
 *          kernel; NULL: one fused product + cell-update kernel per step,
 *          no scratch (slower on large layers).  Both give the same values
 *          up to fp32 summation order. */
int32_t lstm_fwd_cache(const lstmss_dims *d, const void *x, const void *W, const float *b,
                       const float *h0, const float *c0, void *h_out, void *cache, void *ws,
                       size_t ws_bytes, void *stream);

/* Dense backward pass through time of one layer: every gate-gradient row
 * kept, the baseline the paper's speedups are measured against (section 5.5;
 * the dense products of its custom operation, section 4).  Loss convention:
 * dH_up[t] = dL/dh_t from above, dhT, dcT = dL/dh_T, dL/dc_T from later time
 * (NULL = 0).
 *   x, W, cache as given to / written by lstm_fwd_cache
 *   dH_up  [T][H][B] fp32
 *   dX     [T][I][B] fp32 (dL/dx_t), NULL skips the input-gradient rows
 *   dW     [4H][I+H] fp32, overwritten
 *   db     [4H] fp32 or NULL, overwritten
 *   dh0, dc0 [H][B] fp32 (dL/dh_0, dL/dc_0) or NULL
 *   ws     lstmss_workspace_bytes(d, 0, s) bytes (any structure, or NULL s). */
int32_t lstm_bwd_dense(const lstmss_dims *d, const void *x, const void *W, const void *cache,
                       const float *dH_up, const float *dhT, const float *dcT, float *dX,
                       float *dW, float *db, float *dh0, float *dc0, void *ws, size_t ws_bytes,
                       void *stream);

/* Structurally sparsified backward pass (section 3).  COARSE: at every
 * time step the gate gradient is formed, each P-row slice is scored by its
 * squared L2 norm (same ranking as the norm) summed in fp64 in a fixed order
 * (per 64-column batch chunk the squares are combined pairwise by index xor
 * 32, 16, 8, 4, 2, 1; the chunks of a row, then the P rows of a slice, are
 * added in increasing order), the S lowest slices of
 * every region are dropped (ties drop the higher slice index; NaN scores rank
 * highest), the kept rows are compacted in ascending order and both gradient
 * products run on the compacted rows.  The cell-state gradient recursion uses
 * the unsparsified gradient.  With sparsity 0 the result equals
 * lstm_bwd_dense.
 * FINE: every My-column block of an Mx-row slice is scored by its squared L2
 * norm in fp64 (per row, the squares of the block are combined pairwise by
 * column index xor My/2, ..., 2, 1, columns past B adding zero; the Mx rows
 * are added in increasing order), the K lowest blocks of every slice are
 * zeroed (same tie and NaN rules) and the products run on the masked
 * [4H][B] matrix; the kept block indices of slice j are listed ascending.
 * Arguments as lstm_bwd_dense, plus
 *   sparsity, s    structure (see lstmss_structure)
 *   idx_out        [T][lstmss_index_entries] int32 per step (COARSE: kept
 *                  slice indices; FINE: [4H/Mx][nb-K] kept block indices),
 *                  or NULL
 *   dbg_dgates     [T][4H][B] dtype gate gradient before sparsifying (the
 *                  exact values that were scored), or NULL
 *   ws             lstmss_workspace_bytes(d, sparsity, s) bytes. */
int32_t lstm_bwd_structsparse(const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                              const void *x, const void *W, const void *cache,
                              const float *dH_up, const float *dhT, const float *dcT, float *dX,
                              float *dW, float *db, float *dh0, float *dc0, int32_t *idx_out,
                              void *dbg_dgates, void *ws, size_t ws_bytes, void *stream);

/* Score, select and compact one given gate-gradient matrix: the selection
 * step of lstm_bwd_structsparse on its own (section 3: slice scores by L2
 * norm, the S lowest slices of every region dropped, kept slices compacted
 * with an offset index), run by the same kernels the backward pass uses at
 * this shape.
 *   dG     [4H][B] dtype (d->T is ignored)
 *   dG_c   [K'][B] dtype: COARSE kept rows in ascending order; FINE the
 *          masked matrix (removed blocks zero)
 *   idx    [lstmss_index_entries] int32 (see lstm_bwd_structsparse)
 *   scores COARSE [4H/P] fp64 slice scores; FINE [4H/Mx][nb] fp64 block
 *          scores; or NULL
 *   ws     lstmss_select_workspace_bytes(d, sparsity, s) bytes of scratch
 *          (the per-row, per-64-column-chunk sums of squares of the
 *          two-kernel path that the backward pass takes at H*B >= 65536);
 *          may be NULL when that size is 0.  LSTMSS_ERR_WORKSPACE when it is
 *          missing or too small. */
int64_t lstmss_select_workspace_bytes(const lstmss_dims *d, float sparsity,
                                      const lstmss_structure *s);
int32_t lstmss_select_compact(const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                              const void *dG, void *dG_c, int32_t *idx, double *scores, void *ws,
                              size_t ws_bytes, void *stream);

/* lstmss_select_compact without a workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments and results as
 * lstmss_select_compact (bit for bit); the scratch of the two-kernel path
 * (lstmss_select_workspace_bytes, 4H * ceil(B/64) * 8 bytes rounded up to
 * 256) comes from a static device array of LSTMSS_NOALLOC_SCRATCH_BYTES
 * that every GPU the library runs on holds until the process ends.  It
 * allocates nothing and enqueues only the selection kernels; shapes whose
 * scratch exceeds the array return LSTMSS_ERR_UNSUPPORTED before any
 * pointer is used.  All calls on one GPU share that GPU's array (it keeps
 * the last call's contents, which every call overwrites before reading), so
 * calls that overlap in time on one GPU race: serialise them (one stream).
 * Not affected by the timing hooks. */
#define LSTMSS_NOALLOC_SCRATCH_BYTES (1 << 20)
int32_t lstmss_select_compact_noalloc(const lstmss_dims *d, float sparsity,
                                      const lstmss_structure *s, const void *dG, void *dG_c,
                                      int32_t *idx, double *scores, void *stream);

/* Backward pass of a stack of `layers` (1..8) LSTM layers, bottom layer 0,
 * scheduled as a wavefront (the layer-time pipelining of a stacked LSTM):
 * layer l's input gradient dX[l] is layer l-1's upstream gradient, and
 * every layer runs on its own library-owned streams, its step t waiting
 * only for the input-gradient launch of layer l+1 that produced dH_up[t]
 * (launches of LSTMSS_OPT_STACK_DX_STEPS steps), so the layers overlap in
 * time.  Results are those of calling lstm_bwd_structsparse (or, with s
 * NULL or sparsity 0, lstm_bwd_dense) on each layer in turn, top first,
 * with dhT = dcT = NULL.  A stack call of two or more layers is enqueued
 * directly (never recorded into a HIP graph, whatever LSTMSS_OPT_GRAPHS
 * says); a one-layer call is the single-layer call itself.
 *   d            [layers] dims; equal T, B, dtype; d[l].I = d[l-1].H
 *   x, W, cache  [layers] per-layer pointers as for lstm_bwd_structsparse
 *   dH_top       [T][H][B] fp32 upstream gradient of the top layer
 *   dX           [layers] fp32 [T][I_l][B]; dX[0] may be NULL
 *   dW           [layers] fp32 [4H][I_l+H]; db: NULL or [layers] fp32 [4H]
 *                (entries may be NULL)
 *   idx_out      NULL or [layers] (entries may be NULL), as idx_out of
 *                lstm_bwd_structsparse
 *   ws           lstmss_stack_workspace_bytes(...) bytes. */
int64_t lstmss_stack_workspace_bytes(int32_t layers, const lstmss_dims *d, float sparsity,
                                     const lstmss_structure *s);
int32_t lstm_bwd_stack(int32_t layers, const lstmss_dims *d, float sparsity,
                       const lstmss_structure *s, const void *const *x, const void *const *W,
                       const void *const *cache, const float *dH_top, float *const *dX,
                       float *const *dW, float *const *db, int32_t *const *idx_out, void *ws,
                       size_t ws_bytes, void *stream);

/* Bidirectional layer (section 4: the NMT encoder's first layer).  A
 * forward-direction LSTM runs over x_1..x_T and a reverse-direction LSTM,
 * with its own W, over x_T..x_1; the layer's output at time t is
 * [h_fwd_t; h_rev_t] (2H rows).  The reverse direction is an ordinary layer
 * on the time-reversed input x_rev (lstmss_time_reverse, then
 * lstm_fwd_cache), so its cache is in its own processing order.
 * lstmss_time_reverse: dst[s] = src[T-1-s] for T steps of step_bytes bytes
 *   (a positive multiple of 4); src and dst must not overlap.
 * lstmss_bidir_join: out [T][2H][B] dtype, out[t] = [h_fwd[t]; h_rev[T-1-t]]
 *   from the two directions' h_out ([T][H][B] dtype each).
 * lstm_bwd_bidir: the backward pass of both directions, run concurrently on
 *   library-owned streams (enqueued directly, not recorded into a graph).
 *   dH_up [T][2H][B] fp32 is the layer's upstream gradient in time order;
 *   dX [T][I][B] fp32 (or NULL) receives dL/dx_t = the forward direction's
 *   input gradient plus the reverse direction's, mapped back to time order;
 *   dW_*, db_* (db may be NULL), idx_* (may be NULL; the reverse direction's
 *   in its processing order) as for lstm_bwd_structsparse (s NULL or
 *   sparsity 0: dense) for each direction; results equal that call made per
 *   direction on the split upstream gradient.
 *   ws: lstmss_bidir_workspace_bytes(d, sparsity, s) bytes. */
int32_t lstmss_time_reverse(int32_t T, int64_t step_bytes, const void *src, void *dst,
                            void *stream);
int32_t lstmss_bidir_join(const lstmss_dims *d, const void *h_fwd, const void *h_rev, void *out,
                          void *stream);
int64_t lstmss_bidir_workspace_bytes(const lstmss_dims *d, float sparsity,
                                     const lstmss_structure *s);
int32_t lstm_bwd_bidir(const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                       const void *x, const void *x_rev, const void *W_fwd, const void *W_rev,
                       const void *cache_fwd, const void *cache_rev, const float *dH_up, float *dX,
                       float *dW_fwd, float *dW_rev, float *db_fwd, float *db_rev,
                       int32_t *idx_fwd, int32_t *idx_rev, void *ws, size_t ws_bytes,
                       void *stream);

/* Training step pieces around the backward pass (section 4: SGD with a
 * fixed learning rate; section 5: dense-after-sparse schedules).
 * lstmss_sgd_update: W <- W - lr dW (formed in fp32, stored in dtype,
 *   round to nearest even for bf16) and, when b is not NULL, b <- b - lr db.
 *   W [4H][I+H] dtype, dW [4H][I+H] fp32, b, db [4H] fp32.
 * lstmss_mse_grad: regression loss of the top layer's hidden states against
 *   a target, L = (1 / 2B) sum over t, u, n of (h - y)^2:
 *   h [T][H][B] dtype, y [T][H][B] fp32, dH [T][H][B] fp32 = (h - y) / B
 *   (the dH_up of the top layer's backward pass); loss: NULL, or a device
 *   array of LSTMSS_LOSS_SLOTS fp64 values whose last one receives L (the
 *   others hold partial sums), summed in a fixed order. */
#define LSTMSS_LOSS_SLOTS 1025
int32_t lstmss_sgd_update(const lstmss_dims *d, void *W, float *b, const float *dW,
                          const float *db, float lr, void *stream);
int32_t lstmss_mse_grad(const lstmss_dims *d, const void *h, const float *y, float *dH,
                        double *loss, void *stream);

/* Execution options (results are identical under every setting):
 *   LSTMSS_OPT_GRAPHS  1 (default): each backward call's launches are
 *                      captured once into a HIP graph, keyed by every
 *                      argument that reaches a kernel, and replayed on later
 *                      calls with the same arguments (up to 32 per device).
 *                      Environment variable LSTMSS_GRAPHS=0 sets it to 0.
 *   LSTMSS_OPT_SIDE_STREAM  where the work off the sequential critical
 *                      path (weight gradient, input gradient dX) runs:
 *                      0 in order on the caller's stream; 1 on a
 *                      library-owned side stream, overlapping the per-step
 *                      gate kernel and dh GEMM; 2 (default) on the side
 *                      stream while a step's data-gradient GEMM is below
 *                      2^31 multiply-adds ((I+H) * B * K'), else in order
 *                      (large GEMMs fill the GPU by themselves); in stack
 *                      and bidirectional calls mode 2 keeps every layer's
 *                      work in order (the other layers fill the GPU).
 *   LSTMSS_OPT_STACK_DX_STEPS  steps per input-gradient launch inside
 *                      lstm_bwd_stack, i.e. how many steps a layer lags the
 *                      layer above; 0 (default) = 12.
 *   LSTMSS_OPT_FINE_SKIP  FINE with Mx = My = 32 and fp32 storage: 1 (default) skips the
 *                      removed blocks' multiplications, 0 multiplies the
 *                      zeros (same bits; for checking and timing).
 *   LSTMSS_OPT_GEMM_DMA  1 (default): the products load their operand
 *                      tiles from global memory straight into LDS where the
 *                      shape allows (weight gradient: B a multiple of 32 for
 *                      fp32 or 64 for bf16; data gradient and the forward
 *                      products: the contraction length a multiple of 32
 *                      (fp32) or 64 (bf16), rows a multiple of 16 bytes,
 *                      bf16 only with B > 64; the operands 16-byte aligned);
 *                      0 stages them through registers (same bits; for
 *                      checking and timing).
 *   LSTMSS_OPT_GEMM_SELECT  1 (default): on the two-kernel gate path of
 *                      the coarse structure (H * B >= 65536) with DMA data-
 *                      gradient stages, the per-step dh product ranks the
 *                      slices itself (splits of whole regions), reads both
 *                      operands through the kept rows of the element
 *                      kernel's staging matrix and writes the compacted
 *                      matrix and offset index, in place of a separate
 *                      selection launch; 0 always launches the selection
 *                      kernel (same bits; for checking and timing).
 *   LSTMSS_OPT_FINE_FUSED  1 (default): FINE with Mx = 4, H a multiple of 4
 *                      and H * B >= 65536 forms the gate gradient and
 *                      selects the blocks in one kernel per step (each
 *                      work-group holds four whole slices); 0 forms it into
 *                      the staging matrix and selects in a second kernel
 *                      (same bits; for checking and timing).
 *   LSTMSS_OPT_WGRAD_BIG  1 (default): the bf16 weight gradient with 128-byte
 *                      batch chunks (B a multiple of 64, I a multiple of 8)
 *                      runs on 256-row x 256-feature tiles when it is dense
 *                      (sparsity 0 included) or when a coarse structure's
 *                      regions of P * R rows divide 256 and keep 128 or 192
 *                      rows of each tile, with at least 256 tiles; the
 *                      dropped rows are then multiplied as zeros.  0 (and
 *                      every other case) runs the 32-row-group kernel that
 *                      multiplies only the kept rows.  The two sum in
 *                      different orders (both fixed; each matches the oracle
 *                      to the bf16 tolerance).
 * Changing an option drops the recorded graphs.  Not for use while calls
 * are being enqueued from other threads. */
enum {
    LSTMSS_OPT_GRAPHS = 0,
    LSTMSS_OPT_SIDE_STREAM = 1,
    LSTMSS_OPT_STACK_DX_STEPS = 2,
    LSTMSS_OPT_FINE_SKIP = 3,
    LSTMSS_OPT_GEMM_DMA = 4,
    LSTMSS_OPT_GEMM_SELECT = 5,
    LSTMSS_OPT_FINE_FUSED = 6,
    LSTMSS_OPT_WGRAD_BIG = 7
};
int32_t lstmss_set_option(int32_t option, int32_t value);

/* Measurement hooks (not part of the method): when enabled, every kernel the
 * library launches is bracketed by a pair of HIP events recorded on its own
 * launch stream; lstmss_timing_read synchronises on the recorded events and
 * returns the summed event-to-event time and the number of launches of one
 * kernel kind since the last reset.  Timing adds two event records per
 * launch, so leave it off while timing whole calls.  Not for concurrent use
 * from several host threads while enabled. */
enum {
    LSTMSS_KERNEL_GATES = 0,       /* gate gradient + score/select/compact (or dense) */
    LSTMSS_KERNEL_DATA_GRAD = 1,   /* [dx; dh] = W_c^T dG_c, split-K partials */
    LSTMSS_KERNEL_WEIGHT_GRAD = 2, /* dW[kept rows] += dG_c [x; h]^T */
    LSTMSS_KERNEL_AUX = 3,         /* zero fills, final reductions and copies */
    LSTMSS_KERNEL_FORWARD = 4,     /* forward step */
    LSTMSS_KERNEL_KINDS = 5
};
int32_t lstmss_timing_enable(int32_t on);
int32_t lstmss_timing_read(int32_t kind, double *total_ms, int64_t *launches);
int32_t lstmss_timing_reset(void);

#ifdef __cplusplus
}
#endif
#endif /* LSTMSS_H */
