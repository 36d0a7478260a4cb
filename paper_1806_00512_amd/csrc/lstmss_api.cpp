// Host side of liblstmss: argument checks, cache / workspace layout and the
// backward-through-time driver (one layer per call, reverse time loop).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/lstmss.h"
#include "kernels.h"

using namespace lstmss;

namespace {

thread_local std::string g_last_error;

int32_t fail(int32_t code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int32_t fail(int32_t code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

#define HIP_TRY(expr)                                                                          \
    do {                                                                                       \
        hipError_t e_ = (expr);                                                                \
        if (e_ != hipSuccess)                                                                  \
            return fail(LSTMSS_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));        \
    } while (0)

// Optional per-kernel timing with HIP events recorded on the launch stream
// around every kernel of a given kind (enabled by lstmss_timing_enable).
struct TimingRec {
    int kind;
    hipEvent_t a, b;
};
std::mutex g_tmu;
bool g_timing = false;
std::vector<TimingRec> g_pending;
std::vector<hipEvent_t> g_event_pool;
double g_total_ms[LSTMSS_KERNEL_KINDS];
int64_t g_count[LSTMSS_KERNEL_KINDS];

hipEvent_t pooled_event() {
    if (!g_event_pool.empty()) {
        hipEvent_t e = g_event_pool.back();
        g_event_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess)
        return nullptr;
    return e;
}

template <class F>
hipError_t timed(int kind, hipStream_t st, F &&launch) {
    if (!g_timing)
        return launch();
    std::lock_guard<std::mutex> lk(g_tmu);
    hipEvent_t a = pooled_event(), b = pooled_event();
    if (!a || !b)
        return hipErrorOutOfMemory;
    hipError_t e = hipEventRecord(a, st);
    if (e != hipSuccess)
        return e;
    e = launch();
    if (e != hipSuccess)
        return e;
    e = hipEventRecord(b, st);
    g_pending.push_back({kind, a, b});
    return e;
}

// Per-device side stream on which the weight gradient of finished time
// steps runs while the sequential part of the backward pass continues on the
// caller's stream.  Default priority; joined back before each call returns.
constexpr int kMaxWgradChunks = 4;
constexpr int kForkEvents = 8;  // fork points of one call reuse these in turn
struct GraphEntry {
    std::vector<uint64_t> key;
    hipGraphExec_t exec = nullptr;
    uint64_t last_use = 0;
};
struct SideStream {
    hipStream_t s = nullptr;
    hipStream_t cap = nullptr;  // capture stream for graph recording
    hipEvent_t ev[kForkEvents] = {};
    hipEvent_t join = nullptr;
    hipEvent_t fork = nullptr;
    std::vector<GraphEntry> graphs;  // instantiated backward calls, LRU
    uint64_t use_clock = 0;
    std::mutex mu;
};
constexpr size_t kMaxGraphs = 32;
bool g_graphs = true;  // replay captured graphs (LSTMSS_GRAPHS=0 disables)
// off-critical-path work: 0 in order on the caller's stream, 1 on the side
// stream, 2 (default) side stream only while the per-step data-gradient GEMM
// is small (large GEMMs fill the GPU on their own, and overlapping them with
// the critical path only delays it)
int g_side_mode = 2;
constexpr double kSideMaxMacs = 2147483648.0;
std::mutex g_side_mu;
std::map<int, SideStream> g_side;

hipError_t side_stream(SideStream **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    std::lock_guard<std::mutex> lk(g_side_mu);
    SideStream &ss = g_side[dev];
    if (!ss.s) {
        const char *env = getenv("LSTMSS_GRAPHS");
        if (env && env[0] == '0')
            g_graphs = false;
        e = hipStreamCreateWithFlags(&ss.s, hipStreamNonBlocking);
        if (e != hipSuccess)
            return e;
        if ((e = hipStreamCreateWithFlags(&ss.cap, hipStreamNonBlocking)) != hipSuccess)
            return e;
        if ((e = hipEventCreateWithFlags(&ss.fork, hipEventDisableTiming)) != hipSuccess)
            return e;
        for (int i = 0; i < kForkEvents; ++i)
            if ((e = hipEventCreateWithFlags(&ss.ev[i], hipEventDisableTiming)) != hipSuccess)
                return e;
        if ((e = hipEventCreateWithFlags(&ss.join, hipEventDisableTiming)) != hipSuccess)
            return e;
    }
    *out = &ss;
    return hipSuccess;
}

// Streams and events of lstm_bwd_stack (per device): one main and one side
// stream per layer, each layer's fork ring and join event, one event per dX
// chunk per layer.
constexpr int kMaxStackLayers = 8;
struct StackRes {
    hipStream_t main[kMaxStackLayers] = {}, side[kMaxStackLayers] = {};
    hipEvent_t ring[kMaxStackLayers][kForkEvents] = {};
    hipEvent_t join[kMaxStackLayers] = {}, done[kMaxStackLayers] = {};
    hipEvent_t fork = nullptr;
    std::vector<hipEvent_t> chunk_ev[kMaxStackLayers];
#if LSTMSS_STACK_GRAPHS
    // recorded stack calls (LRU), captured on their own stream
    hipStream_t cap = nullptr;
    std::vector<GraphEntry> graphs;
    uint64_t use_clock = 0;
#endif
    std::mutex mu;
};
std::map<int, StackRes> g_stack;
// steps per dX launch inside a stack (the wavefront lag between layers):
// 0 = kStackDxSteps (measured best at T = 35 and T = 50)
int g_stack_dx_steps = 0;
constexpr int kStackDxSteps = 12;
// fine structure with 32 x 32 blocks: skip the removed blocks' products (1,
// default) or run them on the zeros (0); results are the same bits
bool g_fine_skip = true;
bool g_gemm_dma = true;
// coarse selection inside the dh product where the shape allows (1) or in
// its own kernel (0); same bits
bool g_gemm_select = true;
// fine structure with 4-row slices at large shapes: gate gradient and block
// selection in one kernel (1) or two (0); same bits
bool g_fine_fused = true;
// bf16 weight gradient: the 256 x 256-tile kernel where it applies (1) or the
// 32-row-group kernel everywhere (0)
bool g_wgrad_big = true;

hipError_t stack_res(StackRes **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    std::lock_guard<std::mutex> lk(g_side_mu);
    StackRes &r = g_stack[dev];
    if (!r.fork) {
        auto ev = [&](hipEvent_t *q) { return hipEventCreateWithFlags(q, hipEventDisableTiming); };
        for (int l = 0; l < kMaxStackLayers; ++l) {
            if ((e = hipStreamCreateWithFlags(&r.main[l], hipStreamNonBlocking)) != hipSuccess ||
                (e = hipStreamCreateWithFlags(&r.side[l], hipStreamNonBlocking)) != hipSuccess ||
                (e = ev(&r.join[l])) != hipSuccess || (e = ev(&r.done[l])) != hipSuccess)
                return e;
            for (int i = 0; i < kForkEvents; ++i)
                if ((e = ev(&r.ring[l][i])) != hipSuccess)
                    return e;
        }
        if ((e = ev(&r.fork)) != hipSuccess)
            return e;
#if LSTMSS_STACK_GRAPHS
        if ((e = hipStreamCreateWithFlags(&r.cap, hipStreamNonBlocking)) != hipSuccess)
            return e;
#endif
    }
    *out = &r;
    return hipSuccess;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
long ceil_div(long a, long b) { return (a + b - 1) / b; }

// LDS budget of the fused gate-gradient / selection kernel's work-group.
constexpr size_t kMaxLds = 64 * 1024;

int elem_bytes(int32_t dtype) { return dtype == LSTMSS_BF16 ? 2 : 4; }

int32_t check_dims(const lstmss_dims *d) {
    if (!d)
        return fail(LSTMSS_ERR_INVALID_ARG, "dims is NULL");
    if (d->T < 1 || d->B < 1 || d->I < 1 || d->H < 1)
        return fail(LSTMSS_ERR_INVALID_ARG, "dims must be positive (T=%d B=%d I=%d H=%d)", d->T,
                    d->B, d->I, d->H);
    if (d->dtype != LSTMSS_F32 && d->dtype != LSTMSS_BF16)
        return fail(LSTMSS_ERR_UNSUPPORTED, "unknown dtype %d", d->dtype);
    // 32-bit row indices inside the kernels
    if ((int64_t)4 * d->H * ((int64_t)d->I + d->H) >= ((int64_t)1 << 31) ||
        (int64_t)4 * d->H * d->B >= ((int64_t)1 << 31) ||
        ((int64_t)d->I + d->H) * d->B >= ((int64_t)1 << 31) ||
        (int64_t)d->T * 4 * d->H * d->B >= ((int64_t)1 << 40))
        return fail(LSTMSS_ERR_UNSUPPORTED, "sizes too large");
    return LSTMSS_OK;
}

struct Plan {
    int P, R, S;
    long nslices;  // 4H / P
    long kept;     // index entries per step (coarse: kept slices)
    long Kp;       // rows of the products' gate-gradient operand per step
    // fine-grained structure: P = Mx rows per slice, nb blocks of My batch
    // columns, S = K blocks removed per slice; the products then run on the
    // masked [4H][B] matrix (Kp = 4H) and kept = slices * (nb - K)
    bool fine = false;
    int My = 0, nb = 0;
};

// Slices removed from a region of r slices.
long removed(long r, int R, int S) { return (long)S * r / R; }

int32_t make_plan(const lstmss_dims *d, float sparsity, const lstmss_structure *s, bool dense,
                  Plan *p) {
    const long G = 4L * d->H;
    if (dense) {
        p->P = 1;
        p->R = 1;
        p->S = 0;
        p->nslices = G;
        p->kept = G;
        p->Kp = G;
        return LSTMSS_OK;
    }
    if (!s)
        return fail(LSTMSS_ERR_INVALID_ARG, "structure is NULL");
    if (s->kind == LSTMSS_FINE) {
        if (s->Mx < 1 || s->Mx > 32 || G % s->Mx != 0 || 32 % s->Mx != 0)
            return fail(LSTMSS_ERR_INVALID_ARG, "Mx=%d must divide 32 and 4H=%ld", s->Mx, G);
        if (s->My < 2 || s->My > 64 || (s->My & (s->My - 1)) != 0)
            return fail(LSTMSS_ERR_INVALID_ARG, "My=%d must be a power of two in [2, 64]", s->My);
        if (d->B > 256)
            return fail(LSTMSS_ERR_UNSUPPORTED, "fine-grained structure needs B <= 256");
        const long nb = ((long)d->B + s->My - 1) / s->My;
        if (nb > 64)
            return fail(LSTMSS_ERR_INVALID_ARG, "%ld blocks of My=%d per slice (at most 64)", nb,
                        s->My);
        if (!(sparsity >= 0.f) || !(sparsity < 1.f))
            return fail(LSTMSS_ERR_INVALID_ARG, "sparsity %g must be in [0, 1)", (double)sparsity);
        const double kr = (double)sparsity * nb;
        const double Kr = std::nearbyint(kr);
        if (std::fabs(kr - Kr) > 1e-6 * std::fmax(1.0, (double)nb))
            return fail(LSTMSS_ERR_INVALID_ARG, "sparsity %g * %ld blocks is not an integer",
                        (double)sparsity, nb);
        p->fine = true;
        p->P = s->Mx;
        p->My = s->My;
        p->nb = (int)nb;
        p->R = (int)nb;
        p->S = (int)Kr;
        if (p->S < 0 || p->S >= nb)
            return fail(LSTMSS_ERR_INVALID_ARG, "K=%d must be in [0, %ld)", p->S, nb);
        p->nslices = G / s->Mx;
        p->kept = p->nslices * (nb - p->S);
        p->Kp = G;
        return LSTMSS_OK;
    }
    if (s->kind != LSTMSS_COARSE)
        return fail(LSTMSS_ERR_INVALID_ARG, "unknown structure kind %d", s->kind);
    if (s->P < 1 || G % s->P != 0)
        return fail(LSTMSS_ERR_INVALID_ARG, "P=%d must divide 4H=%ld", s->P, G);
    if (s->R < 1 || s->R > 64)
        return fail(LSTMSS_ERR_INVALID_ARG, "R=%d must be in [1, 64]", s->R);
    if (!(sparsity >= 0.f) || !(sparsity < 1.f))
        return fail(LSTMSS_ERR_INVALID_ARG, "sparsity %g must be in [0, 1)", (double)sparsity);
    const double sr = (double)sparsity * s->R;
    const double Sr = std::nearbyint(sr);
    if (std::fabs(sr - Sr) > 1e-6 * std::fmax(1.0, (double)s->R))
        return fail(LSTMSS_ERR_INVALID_ARG, "sparsity %g * R=%d is not an integer", (double)sparsity,
                    s->R);
    const int S = (int)Sr;
    if (S < 0 || S >= s->R)
        return fail(LSTMSS_ERR_INVALID_ARG, "S=%d must be in [0, R)", S);
    p->P = s->P;
    p->R = s->R;
    p->S = S;
    p->nslices = G / s->P;
    const long full = p->nslices / p->R, rest = p->nslices % p->R;
    p->kept = full * (p->R - S) + (rest - removed(rest, p->R, S));
    p->Kp = p->kept * p->P;
    return LSTMSS_OK;
}

struct CacheLayout {
    size_t gates, c, h, total;
};

CacheLayout cache_layout(const lstmss_dims *d) {
    const size_t es = elem_bytes(d->dtype);
    const size_t HB = (size_t)d->H * d->B;
    CacheLayout L;
    L.gates = 0;
    L.c = align256((size_t)d->T * 4 * HB * es);
    L.h = L.c + align256((size_t)(d->T + 1) * HB * 4);
    L.total = L.h + align256((size_t)(d->T + 1) * HB * es);
    return L;
}

// Split of the K' reduction of the critical-path data gradient (the dh rows
// only): enough splits that the 128 x 128 tiles give every CU a work-group
// (fp32) or two (bf16), or, with 64 x 64 tiles, four; each split at least
// two k stages, at most 16 partials for the gate kernel to add up.
int splitk_for(const lstmss_dims *d, long Kp) {
    const bool bf16 = d->dtype == LSTMSS_BF16;
    long target, tiles;
    if (d->B <= 32) {
        tiles = ceil_div(d->H, 128);
        target = 512;
    } else if (d->B <= 64 && !bf16) {
        tiles = ceil_div(d->H, 64);
        target = 1024;
    } else {
        tiles = ceil_div(d->H, 128) * ceil_div(d->B, d->B <= 64 ? 64 : 128);
        target = bf16 ? 512 : 256;
    }
    long sk = ceil_div(target, tiles);
    const long max_sk = std::max(1L, Kp / (2L * GEMM1_TK));
    sk = std::min(std::max(sk, 1L), max_sk);
    return (int)std::min(sk, 16L);
}

// Steps per batched dX launch: whole rounds of the work-groups the GPU holds
// at once (a launch one round too large runs its last few work-groups as a
// nearly empty second round), close to the weight-gradient chunk length.
int dx_chunk_len(const lstmss_dims *d, int chunk_len, int *tm, int *tn) {
    const bool bf16 = d->dtype == LSTMSS_BF16;
    gemm1_tile(bf16, d->B, d->I, 1, tm, tn);
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const long tiles = ceil_div(d->I, *tm) * ceil_div(d->B, *tn);
    const long spr = std::max(1L, (long)cus * gemm1_wgs_per_cu(*tm, *tn) / tiles);
    if (spr >= chunk_len)
        return chunk_len;
    return (int)(spr * std::max(1L, std::lround((double)chunk_len / spr)));
}

struct WsLayout {
    size_t dc0, dc1, part, dGc, idx, db, stage, chunk_sq, chunk_rs, blk, total;
    int splitk;
    long k_chunk;
};

// Bytes of the fine structure's per-step block sums: [4H][nb] doubles, then
// [4H][nb] floats.
size_t blk_sq_bytes(const lstmss_dims *d, const Plan &p) {
    return align256((size_t)4 * d->H * p.nb * 8);
}
size_t blk_bytes(const lstmss_dims *d, const Plan &p) {
    return blk_sq_bytes(d, p) + align256((size_t)4 * d->H * p.nb * 4);
}

WsLayout ws_layout(const lstmss_dims *d, const Plan &p) {
    const size_t es = elem_bytes(d->dtype);
    const size_t HB = (size_t)d->H * d->B;
    WsLayout L;
    L.splitk = splitk_for(d, p.Kp);
    L.k_chunk = ceil_div(ceil_div(p.Kp, L.splitk), GEMM1_TK) * GEMM1_TK;
    L.splitk = (int)ceil_div(p.Kp, L.k_chunk);
    size_t off = 0;
    L.dc0 = off; off += align256(HB * 4);
    L.dc1 = off; off += align256(HB * 4);
    L.part = off; off += align256((size_t)L.splitk * HB * 4);
    L.dGc = off; off += align256((size_t)d->T * p.Kp * d->B * es);
    L.idx = off; off += align256((size_t)d->T * p.kept * 4);
    L.db = off; off += align256((size_t)4 * d->H * 4);
    // split gate-kernel path: staging matrix, chunk sums of one step, chunk
    // row sums of every step (for the bias gradient)
    const size_t nch = (size_t)ceil_div(d->B, 64);
    L.stage = off; off += align256((size_t)4 * d->H * d->B * es);
    L.chunk_sq = off; off += align256((size_t)4 * d->H * nch * 8);
    L.chunk_rs = off; off += align256((size_t)d->T * 4 * d->H * nch * 4);
    // fine structure: per (row, block) sums of squares (fp64) and sums (fp32)
    // of one step
    L.blk = off; off += p.fine ? blk_bytes(d, p) : 0;
    L.total = off;
    return L;
}

// Scratch of the standalone selection: the per-(row, 64-column chunk) sums of
// squares of the element kernel when the shape takes the two-kernel path of
// the backward pass (coarse structure), else nothing.
size_t select_ws_bytes(const lstmss_dims *d, const Plan &p) {
    if (p.fine)
        return 0;
    CellArgs probe{};
    probe.B = d->B; probe.H = d->H; probe.P = p.P; probe.R = p.R;
    probe.regions_per_wg = std::max(1, 32 / (p.R * p.P));
    if (!cell_split_ok(probe, CELL_GIVEN))
        return 0;
    return align256((size_t)4 * d->H * ceil_div(d->B, 64) * 8);
}

// Streams and events one backward call is enqueued with.  In a layer stack
// (lstm_bwd_stack) a layer's step t waits for the dX chunk of the layer above
// that holds its upstream gradient dH_up[t], and records an event after each
// of its own dX chunks for the layer below.
struct ChunkEv {
    int t_lo, t_hi;  // steps [t_lo, t_hi)
    hipEvent_t ev;   // recorded after the chunk's launch
};
struct EnqCtx {
    hipStream_t side = nullptr;                      // off-critical-path work
    hipEvent_t *ring = nullptr;                      // fork events, used in turn
    int nring = 0;
    hipEvent_t join = nullptr;                       // side -> main at the end
    const std::vector<ChunkEv> *dH_ready = nullptr;  // chunks of the layer above
    std::vector<ChunkEv> *dx_done = nullptr;         // this layer's dX chunks
    std::vector<hipEvent_t> *dx_events = nullptr;    // events for them (one per chunk)
    int max_dx_len = 0;                              // cap on steps per dX launch (0: none)
    // automatic side-stream mode may use the side stream (single calls);
    // calls that run beside other layers (stack, bidirectional) keep their
    // work in order unless the side stream is forced
    bool auto_side = true;
};

// Whether the coarse structure's gate path splits into the element kernel
// and a selection (large shapes), and whether that selection then runs
// inside the per-step dh product (LSTMSS_OPT_GEMM_SELECT, DMA stages, splits
// of whole regions).  W, ws: the call's weight and workspace pointers (their
// alignment decides the DMA stages).
struct GatePath {
    bool split, select_in_product;
};

GatePath gate_path(const lstmss_dims *d, const Plan &p, bool dense, const void *W, const void *ws) {
    const bool sparse = !dense, fine = sparse && p.fine, gsparse = sparse && !fine;
    CellArgs probe{};
    probe.B = d->B; probe.H = d->H; probe.P = sparse ? p.P : 1; probe.R = sparse ? p.R : 1;
    probe.regions_per_wg = sparse ? std::max(1, 32 / (p.R * p.P)) : 32;
    GatePath g;
    g.split = !fine && cell_split_ok(probe, sparse ? CELL_SPARSE : CELL_DENSE);
    g.select_in_product = false;
    if (!g.split || !gsparse || !g_gemm_select)
        return g;
    const WsLayout L = ws_layout(d, p);
    const long K = (long)d->I + d->H;
    const char *wb = (const char *)ws;
    Gemm1Args a{};
    a.W = W; a.ldw = K; a.P = p.P; a.Kp = p.Kp; a.M = (int)K; a.m_begin = d->I; a.N = d->B;
    a.out_row0 = d->I; a.splitk = L.splitk; a.k_chunk = L.k_chunk; a.steps = 1;
    a.dma = g_gemm_dma ? 1 : 0;
    a.Gc = wb + L.stage;
    a.sel_sq = (const double *)(wb + L.chunk_sq);
    a.sel_nch = (int)ceil_div(d->B, 64); a.sel_R = p.R; a.sel_S = p.S; a.sel_nslices = p.nslices;
    a.sel_gc = const_cast<char *>(wb + L.dGc);
    a.sel_idx = (int32_t *)const_cast<char *>(wb + L.idx);
    // every step's compacted matrix starts Kp * B elements after the last
    if (((size_t)p.Kp * d->B * elem_bytes(d->dtype)) % 16 != 0)
        return g;
    g.select_in_product = gemm1_select_ok(a, d->dtype == LSTMSS_BF16);
    return g;
}

// Enqueue one backward call on main stream st, with ctx (locked by the
// caller) for the off-critical-path work.  Arguments already checked.
int32_t backward_enqueue(const lstmss_dims *d, bool dense, const Plan &p, const void *x,
                         const void *W, const void *cache, const float *dH_up, const float *dhT,
                         const float *dcT, float *dX, float *dW, float *db, float *dh0,
                         float *dc0, int32_t *idx_out, void *dbg, void *ws, hipStream_t st,
                         const EnqCtx &ctx) {
    const WsLayout L = ws_layout(d, p);
    const bool bf16 = d->dtype == LSTMSS_BF16;
    const bool sparse = !dense;
    // the fine structure masks the gate gradient in place; its products run
    // on the masked matrix like the dense ones, without a row gather
    const bool fine = sparse && p.fine;
    const bool gsparse = sparse && !fine;
    // fine blocks shaped like the MFMA operand blocks (32 gate rows x 32
    // batch columns): the products skip the removed blocks
    // batch chunks of 32 columns: the weight gradient takes this path (with or
    // without skipping) whenever the blocks are 32 x 32, so that its
    // summation order does not depend on the skip option.  fp32 only: the
    // bf16 products are bound by their loads, and the dense kernels on the
    // masked matrix measured faster than skipping there
    const bool fblocks = fine && d->dtype == LSTMSS_F32 && p.P == 32 && p.My == 32 &&
                         d->B % 32 == 0 && 4L * d->H / 32 <= FINE_MAX_SLICES;
    const bool ffast = fblocks && g_fine_skip;
    const int fkept = fine ? p.nb - p.S : 0;
    const int T = d->T, B = d->B, I = d->I, H = d->H;
    const long HB = (long)H * B, G = 4L * H, K = (long)I + H;
    const size_t es = elem_bytes(d->dtype);
    const CacheLayout C = cache_layout(d);
    const char *cb = (const char *)cache;
    const char *gates = cb + C.gates;
    const float *cst = (const float *)(cb + C.c);
    const char *hst = cb + C.h;
    char *wb = (char *)ws;
    float *dcbuf[2] = {(float *)(wb + L.dc0), (float *)(wb + L.dc1)};
    float *part = (float *)(wb + L.part);
    char *dGc_all = wb + L.dGc;
    int32_t *idx_all = idx_out ? idx_out : (int32_t *)(wb + L.idx);
    float *dbp = db ? db : (float *)(wb + L.db);

    // Work off the sequential critical path runs on a side stream, in chunks
    // of time steps launched as soon as the gate gradients of their steps
    // exist: the weight gradient (one batched launch per chunk when the
    // structure fits its routing tiles, else a per-step accumulation on the
    // main stream) and the input gradient dX (a batched data-gradient GEMM
    // over the chunk's steps).  The main stream only carries the gate kernel
    // and the dh rows of the data gradient for every step.
    const bool batched = !gsparse || wgrad_supported(p.P, p.R, p.S);
    if (!batched)
        HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] { return launch_fill(dW, G * K, 0.f, st); }));
    // gate kernels: the split path (large shapes) leaves the bias gradient to
    // one kernel after the time loop; the single-kernel paths accumulate it
    const GatePath gp = gate_path(d, p, dense, W, ws);
    const bool split = gp.split;
    const int nch = (int)ceil_div(B, 64);
    float *chunk_rs_all = (float *)(wb + L.chunk_rs);
    if (!split)
        HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] { return launch_fill(dbp, G, 0.f, st); }));

    const bool use_side = batched || dX;
    const bool concurrent = use_side && (g_side_mode == 1 ||
                                         (g_side_mode == 2 && ctx.auto_side &&
                                          (double)K * B * p.Kp < kSideMaxMacs));
    hipStream_t sst = concurrent ? ctx.side : st;
    // the weight gradient runs in chunks of chunk_len steps and dX in chunks
    // of dx_len steps (whole rounds of resident work-groups); each launches
    // once its lowest step has its gate gradients
    int chunk_len = T, dx_len = T, dx_tm = 0, dx_tn = 0;
    if (use_side) {
        // in order on the main stream one weight-gradient launch covers the
        // whole call (dW written once); on the side stream chunks of steps
        // start as soon as their gate gradients exist
        const int nchunks = concurrent ? std::max(1, std::min(kMaxWgradChunks, T / 8)) : 1;
        chunk_len = (int)ceil_div(T, nchunks);
        if (dX)
            dx_len = dx_chunk_len(d, chunk_len, &dx_tm, &dx_tn);
        if (dX && ctx.max_dx_len > 0 && dx_len > ctx.max_dx_len)
            dx_len = ctx.max_dx_len;
    }
    int wg_hi = T, dx_hi = T, wg_count = 0, forks = 0;
    WgradArgs wg{};
    wg.Gc = dGc_all; wg.idx = gsparse ? idx_all : nullptr; wg.x = x; wg.h = hst;
    wg.T = T; wg.I = I; wg.H = H; wg.B = B; wg.Kp = (int)p.Kp; wg.kept = (int)p.kept;
    wg.P = p.P; wg.R = p.R; wg.S = p.S; wg.dW = dW;
    wg.fidx = fblocks ? idx_all : nullptr; wg.fkept = fkept; wg.fskip = ffast ? 1 : 0;
    wg.dma = g_gemm_dma ? 1 : 0;
    wg.big = g_wgrad_big ? 1 : 0;

    Gemm1Args gx{};  // dX[t] = (W_c rows [0, I))^T dG_c, several steps per launch
    gx.W = W; gx.ldw = K; gx.P = p.P; gx.Kp = p.Kp; gx.M = I; gx.m_begin = 0; gx.N = B;
    gx.out_row0 = 0; gx.part_stride = 0; gx.splitk = 1;
    gx.k_chunk = ceil_div(p.Kp, GEMM1_TK) * GEMM1_TK;
    gx.gc_step = p.Kp * B; gx.idx_step = p.kept; gx.out_step = (long)I * B;
    gx.tm = dx_tm; gx.tn = dx_tn;
    gx.fkept = fkept; gx.fidx_step = p.kept;
    gx.dma = g_gemm_dma ? 1 : 0;

    const long part_stride = HB;
    // dh rows of the data gradient for the next (earlier) step
    Gemm1Args g1{};
    g1.W = W; g1.ldw = K; g1.P = p.P;
    g1.Kp = p.Kp; g1.M = (int)K; g1.m_begin = I; g1.N = B; g1.out_row0 = I;
    g1.part = part; g1.part_stride = part_stride; g1.splitk = L.splitk;
    g1.k_chunk = L.k_chunk; g1.steps = 1;
    g1.fkept = fkept; g1.fidx_step = p.kept;
    g1.dma = g_gemm_dma ? 1 : 0;
    // coarse structure on the two-kernel gate path: the dh product selects
    // (from the element kernel's chunk sums) and compacts, so no selection
    // kernel runs between the two; the off-path work of a step is then
    // forked after the product, which writes its compacted rows and index
    const bool sel_gemm = gp.select_in_product;
    auto launch_dh = [&](char *dGc, int32_t *idx) -> int32_t {
        if (sel_gemm) {
            g1.Gc = wb + L.stage; g1.idx = nullptr;
            g1.sel_sq = (const double *)(wb + L.chunk_sq);
            g1.sel_nch = nch; g1.sel_R = p.R; g1.sel_S = p.S; g1.sel_nslices = p.nslices;
            g1.sel_gc = dGc; g1.sel_idx = idx;
        } else {
            g1.Gc = dGc; g1.idx = gsparse ? idx : nullptr;
        }
        g1.fidx = ffast ? idx : nullptr;
        HIP_TRY(timed(LSTMSS_KERNEL_DATA_GRAD, st, [&] { return launch_gemm1(g1, bf16, st); }));
        return LSTMSS_OK;
    };
    for (int t = T - 1; t >= 0; --t) {
        const bool last = t == T - 1;
        char *dGc = dGc_all + (size_t)t * p.Kp * B * es;
        int32_t *idx = idx_all + (size_t)t * p.kept;

        if (ctx.dH_ready)  // upstream gradient of this step from the layer above
            for (const ChunkEv &c : *ctx.dH_ready)
                if (c.t_hi - 1 == t)
                    HIP_TRY(hipStreamWaitEvent(st, c.ev, 0));

        CellArgs ca{};
        ca.B = B; ca.H = H; ca.I = I;
        ca.P = sparse ? p.P : 1; ca.R = sparse ? p.R : 1; ca.S = sparse ? p.S : 0;
        ca.nslices = sparse ? p.nslices : G;
        if (sparse)
            ca.regions_per_wg = std::max(1, 32 / (p.R * p.P));
        else
            ca.regions_per_wg = 32;  // dense: 32 rows per work-group
        ca.gates = gates + (size_t)t * G * B * es;
        ca.c_t = cst + (size_t)(t + 1) * HB;
        ca.c_prev = cst + (size_t)t * HB;
        ca.dH_up = dH_up + (size_t)t * HB;
        if (last) {
            ca.dh_part = dhT;
            ca.dh_nparts = dhT ? 1 : 0;
            ca.dh_stride = 0;
            ca.dc_in = dcT;
        } else {
            ca.dh_part = part;
            ca.dh_nparts = L.splitk;
            ca.dh_stride = part_stride;
            ca.dc_in = dcbuf[(t + 1) & 1];
        }
        ca.dc_out = dcbuf[t & 1];
        ca.dGc = dGc;
        ca.idx = sparse ? idx : nullptr;
        ca.db = dbp;
        ca.dbg = dbg ? (char *)dbg + (size_t)t * G * B * es : nullptr;
        ca.scores = nullptr;
        if (split || fine) {
            // staging matrix of the element kernel (used by the fine
            // structure's large-shape path too, which keeps db in its
            // selection kernel)
            ca.stage = wb + L.stage;
            ca.chunk_sq = (double *)(wb + L.chunk_sq);
            ca.chunk_rs = chunk_rs_all + (size_t)t * G * nch;
        }
        if (split)
            ca.db = nullptr;
        ca.defer_select = sel_gemm ? 1 : 0;
        ca.My = p.My;
        ca.nb = p.nb;
        ca.fine_fused = g_fine_fused ? 1 : 0;
        if (fine) {
            ca.blk_sq = (double *)(wb + L.blk);
            ca.blk_rs = (float *)(wb + L.blk + blk_sq_bytes(d, p));
        }
        if (!split && !fine &&
            cell_lds_bytes(ca, sparse ? CELL_SPARSE : CELL_DENSE) > kMaxLds)
            return fail(LSTMSS_ERR_UNSUPPORTED, "R*P*B too large for one work-group's LDS");
        HIP_TRY(timed(LSTMSS_KERNEL_GATES, st, [&] {
            return fine ? launch_cell_fine(ca, CELL_SPARSE, bf16, st)
                        : launch_cell(ca, sparse ? CELL_SPARSE : CELL_DENSE, bf16, st);
        }));

        if (sel_gemm) {
            const int32_t rc = launch_dh(dGc, idx);
            if (rc)
                return rc;
        }

        const bool wg_now = use_side && batched && t == std::max(0, wg_hi - chunk_len);
        const bool dx_now = use_side && dX && t == std::max(0, dx_hi - dx_len);
        if ((wg_now || dx_now) && concurrent) {
            hipEvent_t e = ctx.ring[forks++ % ctx.nring];
            HIP_TRY(hipEventRecord(e, st));
            HIP_TRY(hipStreamWaitEvent(ctx.side, e, 0));
        }
        if (wg_now) {
            wg.t_begin = t;
            wg.t_end = wg_hi;
            wg.accumulate = wg_count++ > 0;
            HIP_TRY(timed(LSTMSS_KERNEL_WEIGHT_GRAD, sst, [&] { return launch_wgrad(wg, gsparse, bf16, sst); }));
            wg_hi = t;
        }
        if (dx_now) {
            gx.Gc = dGc;
            gx.idx = gsparse ? idx : nullptr;
            gx.fidx = ffast ? idx : nullptr;
            gx.part = dX + (size_t)t * I * B;
            gx.steps = dx_hi - t;
            HIP_TRY(timed(LSTMSS_KERNEL_DATA_GRAD, sst, [&] { return launch_gemm1(gx, bf16, sst); }));
            if (ctx.dx_done) {
                const size_t k = ctx.dx_done->size();
                if (k >= ctx.dx_events->size())
                    return fail(LSTMSS_ERR_HIP, "too few chunk events");
                HIP_TRY(hipEventRecord((*ctx.dx_events)[k], sst));
                ctx.dx_done->push_back(ChunkEv{t, dx_hi, (*ctx.dx_events)[k]});
            }
            dx_hi = t;
        }

        if (!sel_gemm) {
            const int32_t rc = launch_dh(dGc, idx);
            if (rc)
                return rc;
        }

        if (!batched) {
            Gemm2Args g2{};
            g2.Gc = dGc; g2.idx = gsparse ? idx : nullptr; g2.P = p.P; g2.Kp = p.Kp;
            g2.xt = (const char *)x + (size_t)t * I * B * es;
            g2.hp = hst + (size_t)t * HB * es;
            g2.I = I; g2.H = H; g2.B = B; g2.dW = dW;
            HIP_TRY(timed(LSTMSS_KERNEL_WEIGHT_GRAD, st, [&] { return launch_gemm2(g2, bf16, st); }));
        }
    }
    if (concurrent) {
        HIP_TRY(hipEventRecord(ctx.join, ctx.side));
        HIP_TRY(hipStreamWaitEvent(st, ctx.join, 0));
    }
    if (split)
        HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] {
            return launch_bias_grad(dbp, chunk_rs_all, nch, G, 0, T, sparse ? idx_all : nullptr,
                                    (int)p.kept, p.P, p.R, p.S, false, st);
        }));
    if (dh0)
        HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] { return launch_reduce_parts(dh0, part, L.splitk, part_stride, HB, st); }));
    if (dc0)
        HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] { return launch_copy_in(dc0, dcbuf[0], HB, st); }));
    return LSTMSS_OK;
}

// A backward call is a fixed DAG of launches for given arguments, so it is
// captured once into a HIP graph (main and side streams joined by events)
// and replayed; the key is every argument that reaches a kernel.
int32_t backward(const lstmss_dims *d, bool dense, float sparsity, const lstmss_structure *s,
                 const void *x, const void *W, const void *cache, const float *dH_up,
                 const float *dhT, const float *dcT, float *dX, float *dW, float *db, float *dh0,
                 float *dc0, int32_t *idx_out, void *dbg, void *ws, size_t ws_bytes,
                 void *stream) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    Plan p;
    rc = make_plan(d, sparsity, s, dense, &p);
    if (rc)
        return rc;
    if (!x || !W || !cache || !dH_up || !dW || !ws)
        return fail(LSTMSS_ERR_INVALID_ARG, "a required pointer is NULL");
    const WsLayout L = ws_layout(d, p);
    if (ws_bytes < L.total)
        return fail(LSTMSS_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", ws_bytes, L.total);
    hipStream_t st = (hipStream_t)stream;
    SideStream *side = nullptr;
    HIP_TRY(side_stream(&side));
    std::unique_lock<std::mutex> lk(side->mu);
    bool timing;
    {
        std::lock_guard<std::mutex> tl(g_tmu);
        timing = g_timing;
    }
    EnqCtx ctx;
    ctx.side = side->s;
    ctx.ring = side->ev;
    ctx.nring = kForkEvents;
    ctx.join = side->join;
    if (!g_graphs || timing)
        return backward_enqueue(d, dense, p, x, W, cache, dH_up, dhT, dcT, dX, dW, db, dh0, dc0,
                                idx_out, dbg, ws, st, ctx);

    auto u = [](const void *q) { return (uint64_t)(uintptr_t)q; };
    std::vector<uint64_t> key = {(uint64_t)d->T, (uint64_t)d->B, (uint64_t)d->I, (uint64_t)d->H,
                                 (uint64_t)d->dtype, (uint64_t)dense, (uint64_t)p.P,
                                 (uint64_t)p.R, (uint64_t)p.S, (uint64_t)p.fine, (uint64_t)p.My,
                                 u(x), u(W), u(cache), u(dH_up),
                                 u(dhT), u(dcT), u(dX), u(dW), u(db), u(dh0), u(dc0), u(idx_out),
                                 u(dbg), u(ws)};
    GraphEntry *hit = nullptr;
    for (GraphEntry &g : side->graphs)
        if (g.key == key)
            hit = &g;
    if (!hit) {
        // record on the private capture stream; the side stream joins the
        // capture through the fork/join events inside backward_enqueue
        HIP_TRY(hipStreamBeginCapture(side->cap, hipStreamCaptureModeRelaxed));
        rc = backward_enqueue(d, dense, p, x, W, cache, dH_up, dhT, dcT, dX, dW, db, dh0, dc0,
                              idx_out, dbg, ws, side->cap, ctx);
        hipGraph_t graph = nullptr;
        const hipError_t ec = hipStreamEndCapture(side->cap, &graph);
        if (rc != LSTMSS_OK) {
            if (graph)
                (void)hipGraphDestroy(graph);
            return rc;
        }
        if (ec != hipSuccess)
            return fail(LSTMSS_ERR_HIP, "graph capture failed: %s", hipGetErrorString(ec));
        hipGraphExec_t exec = nullptr;
        const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
        (void)hipGraphDestroy(graph);
        if (ei != hipSuccess)
            return fail(LSTMSS_ERR_HIP, "graph instantiation failed: %s", hipGetErrorString(ei));
        if (side->graphs.size() >= kMaxGraphs) {
            size_t oldest = 0;
            for (size_t i = 1; i < side->graphs.size(); ++i)
                if (side->graphs[i].last_use < side->graphs[oldest].last_use)
                    oldest = i;
            (void)hipGraphExecDestroy(side->graphs[oldest].exec);
            side->graphs.erase(side->graphs.begin() + oldest);
        }
        side->graphs.push_back(GraphEntry{key, exec, 0});
        hit = &side->graphs.back();
    }
    hit->last_use = ++side->use_clock;
    HIP_TRY(hipGraphLaunch(hit->exec, st));
    return LSTMSS_OK;
}

struct StackPlan {
    std::vector<Plan> plans;
    std::vector<size_t> ws_off;
    size_t total = 0;
    bool dense = true;
};

int32_t stack_plan(int32_t layers, const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                   StackPlan *sp) {
    if (layers < 1 || layers > kMaxStackLayers)
        return fail(LSTMSS_ERR_INVALID_ARG, "layers=%d must be in [1, %d]", layers,
                    kMaxStackLayers);
    if (!d)
        return fail(LSTMSS_ERR_INVALID_ARG, "dims is NULL");
    sp->dense = s == nullptr || sparsity == 0.f;
    sp->plans.assign(layers, Plan{});
    sp->ws_off.assign(layers, 0);
    sp->total = 0;
    for (int l = 0; l < layers; ++l) {
        int32_t rc = check_dims(&d[l]);
        if (rc)
            return rc;
        if (d[l].T != d[0].T || d[l].B != d[0].B || d[l].dtype != d[0].dtype)
            return fail(LSTMSS_ERR_INVALID_ARG, "layer %d: T, B and dtype must match layer 0", l);
        if (l > 0 && d[l].I != d[l - 1].H)
            return fail(LSTMSS_ERR_INVALID_ARG, "layer %d: I=%d must equal the H=%d below", l,
                        d[l].I, d[l - 1].H);
        rc = make_plan(&d[l], sparsity, s, sp->dense, &sp->plans[l]);
        if (rc)
            return rc;
        sp->ws_off[l] = sp->total;
        sp->total += align256(ws_layout(&d[l], sp->plans[l]).total);
    }
    return LSTMSS_OK;
}

// Wavefront backward of a layer stack: every layer runs on its own pair of
// streams; layer l's step t waits only for the dX chunk of layer l + 1 that
// holds its dH_up[t], so the layers overlap in time, each lagging the one
// above by one dX chunk.
int32_t stack_enqueue(int32_t layers, const lstmss_dims *d, const StackPlan &sp,
                      const void *const *x, const void *const *W, const void *const *cache,
                      const float *dH_top, float *const *dX, float *const *dW, float *const *db,
                      int32_t *const *idx_out, void *ws, hipStream_t origin, StackRes &R) {
    std::vector<ChunkEv> chunks[kMaxStackLayers];
    HIP_TRY(hipEventRecord(R.fork, origin));
    for (int l = layers - 1; l >= 0; --l) {
        hipStream_t ms = R.main[l];
        HIP_TRY(hipStreamWaitEvent(ms, R.fork, 0));
        EnqCtx ctx;
        ctx.side = R.side[l];
        ctx.ring = R.ring[l];
        ctx.nring = kForkEvents;
        ctx.join = R.join[l];
        ctx.dH_ready = l == layers - 1 ? nullptr : &chunks[l + 1];
        ctx.dx_done = l > 0 ? &chunks[l] : nullptr;
        ctx.dx_events = &R.chunk_ev[l];
        ctx.max_dx_len = g_stack_dx_steps > 0 ? g_stack_dx_steps : kStackDxSteps;
        ctx.auto_side = false;
        const float *up = l == layers - 1 ? dH_top : dX[l + 1];
        const int32_t rc = backward_enqueue(&d[l], sp.dense, sp.plans[l], x[l], W[l], cache[l],
                                            up, nullptr, nullptr, dX[l], dW[l], db ? db[l] : nullptr,
                                            nullptr, nullptr, idx_out ? idx_out[l] : nullptr,
                                            nullptr, (char *)ws + sp.ws_off[l], ms, ctx);
        if (rc != LSTMSS_OK)
            return rc;
        HIP_TRY(hipEventRecord(R.done[l], ms));
        HIP_TRY(hipStreamWaitEvent(origin, R.done[l], 0));
    }
    return LSTMSS_OK;
}

struct BidirLayout {
    size_t ws_f, ws_r, dh_f, dh_r, dx_f, dx_r, total;
};

BidirLayout bidir_layout(const lstmss_dims *d, const Plan &p) {
    BidirLayout B;
    const size_t one = align256(ws_layout(d, p).total);
    const size_t hb = align256((size_t)d->T * d->H * d->B * 4);
    const size_t ib = align256((size_t)d->T * d->I * d->B * 4);
    B.ws_f = 0;
    B.ws_r = one;
    B.dh_f = 2 * one;
    B.dh_r = B.dh_f + hb;
    B.dx_f = B.dh_r + hb;
    B.dx_r = B.dx_f + ib;
    B.total = B.dx_r + ib;
    return B;
}

// Both directions of a bidirectional layer on their own stream pairs; the
// upstream gradient is split (the reverse half reversed in time) first and
// the input gradients are summed (the reverse one reversed back) last.
int32_t bidir_enqueue(const lstmss_dims *d, bool dense, const Plan &p, const void *x,
                      const void *x_rev, const void *W_f, const void *W_r, const void *cache_f,
                      const void *cache_r, const float *dH_up, float *dX, float *dW_f,
                      float *dW_r, float *db_f, float *db_r, int32_t *idx_f, int32_t *idx_r,
                      void *ws, hipStream_t origin, StackRes &R) {
    const BidirLayout Lb = bidir_layout(d, p);
    char *wb = (char *)ws;
    float *dh_f = (float *)(wb + Lb.dh_f), *dh_r = (float *)(wb + Lb.dh_r);
    float *dx_f = dX ? (float *)(wb + Lb.dx_f) : nullptr;
    float *dx_r = dX ? (float *)(wb + Lb.dx_r) : nullptr;
    const long HB = (long)d->H * d->B, IB = (long)d->I * d->B;
    HIP_TRY(timed(LSTMSS_KERNEL_AUX, origin, [&] {
        return launch_bidir_split(dH_up, dh_f, dh_r, d->T, HB, origin);
    }));
    HIP_TRY(hipEventRecord(R.fork, origin));
    for (int dir = 0; dir < 2; ++dir) {
        hipStream_t ms = R.main[dir];
        HIP_TRY(hipStreamWaitEvent(ms, R.fork, 0));
        EnqCtx ctx;
        ctx.side = R.side[dir];
        ctx.ring = R.ring[dir];
        ctx.nring = kForkEvents;
        ctx.join = R.join[dir];
        ctx.auto_side = false;
        const int32_t rc =
            dir == 0 ? backward_enqueue(d, dense, p, x, W_f, cache_f, dh_f, nullptr, nullptr, dx_f,
                                        dW_f, db_f, nullptr, nullptr, idx_f, nullptr,
                                        wb + Lb.ws_f, ms, ctx)
                     : backward_enqueue(d, dense, p, x_rev, W_r, cache_r, dh_r, nullptr, nullptr,
                                        dx_r, dW_r, db_r, nullptr, nullptr, idx_r, nullptr,
                                        wb + Lb.ws_r, ms, ctx);
        if (rc != LSTMSS_OK)
            return rc;
        HIP_TRY(hipEventRecord(R.done[dir], ms));
        HIP_TRY(hipStreamWaitEvent(origin, R.done[dir], 0));
    }
    if (dX)
        HIP_TRY(timed(LSTMSS_KERNEL_AUX, origin, [&] {
            return launch_sum_rev(dx_f, dx_r, dX, d->T, IB, origin);
        }));
    return LSTMSS_OK;
}

} // namespace

namespace lstmss {

int32_t set_error(int32_t code, const char *msg) { return fail(code, "%s", msg); }

int64_t select_scratch_bytes(const lstmss_dims *d, float sparsity, const lstmss_structure *s) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    Plan p;
    rc = make_plan(d, sparsity, s, false, &p);
    if (rc)
        return rc;
    return (int64_t)select_ws_bytes(d, p);
}

// The standalone selection (lstmss_select_compact); `hooks` false skips the
// timing hooks (whose event pool may create events), for the entry point
// that must not allocate.
int32_t select_compact_impl(const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                            const void *dG, void *dG_c, int32_t *idx, double *scores, void *ws,
                            size_t ws_bytes, void *stream, bool hooks) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    Plan p;
    rc = make_plan(d, sparsity, s, false, &p);
    if (rc)
        return rc;
    if (!dG || !dG_c || !idx)
        return fail(LSTMSS_ERR_INVALID_ARG, "a required pointer is NULL");
    const size_t need = select_ws_bytes(d, p);
    if (need > 0 && (!ws || ws_bytes < need))
        return fail(LSTMSS_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", ws ? ws_bytes : 0,
                    need);
    CellArgs ca{};
    ca.B = d->B; ca.H = d->H; ca.I = d->I;
    ca.P = p.P; ca.R = p.R; ca.S = p.S;
    ca.nslices = p.nslices;
    ca.regions_per_wg = std::max(1, 32 / (p.R * p.P));
    ca.dG_in = dG;
    ca.dGc = dG_c;
    ca.idx = idx;
    ca.scores = scores;
    ca.My = p.My;
    ca.nb = p.nb;
    if (p.fine) {
        hipStream_t st = (hipStream_t)stream;
        auto go = [&] { return launch_cell_fine(ca, CELL_GIVEN, d->dtype == LSTMSS_BF16, st); };
        HIP_TRY(hooks ? timed(LSTMSS_KERNEL_GATES, st, go) : go());
        return LSTMSS_OK;
    }
    if (need > 0)  // the two-kernel path of the backward pass at this shape
        ca.chunk_sq = (double *)ws;
    else if (cell_lds_bytes(ca, CELL_GIVEN) > kMaxLds)
        return fail(LSTMSS_ERR_UNSUPPORTED, "R*P*B too large for one work-group's LDS");
    hipStream_t st = (hipStream_t)stream;
    auto go = [&] { return launch_cell(ca, CELL_GIVEN, d->dtype == LSTMSS_BF16, st); };
    HIP_TRY(hooks ? timed(LSTMSS_KERNEL_GATES, st, go) : go());
    return LSTMSS_OK;
}

} // namespace lstmss

extern "C" {

int32_t lstmss_time_reverse(int32_t T, int64_t step_bytes, const void *src, void *dst,
                            void *stream) {
    if (T < 1 || step_bytes <= 0 || step_bytes % 4 != 0)
        return fail(LSTMSS_ERR_INVALID_ARG, "T=%d, step_bytes=%lld (a positive multiple of 4)",
                    T, (long long)step_bytes);
    if (!src || !dst || src == dst)
        return fail(LSTMSS_ERR_INVALID_ARG, "src and dst must be distinct non-NULL buffers");
    hipStream_t st = (hipStream_t)stream;
    HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] { return launch_reverse(src, dst, T, step_bytes / 4, st); }));
    return LSTMSS_OK;
}

int32_t lstmss_bidir_join(const lstmss_dims *d, const void *h_fwd, const void *h_rev, void *out,
                          void *stream) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    if (!h_fwd || !h_rev || !out)
        return fail(LSTMSS_ERR_INVALID_ARG, "a required pointer is NULL");
    hipStream_t st = (hipStream_t)stream;
    HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] {
        return launch_bidir_join(h_fwd, h_rev, out, d->T, (long)d->H * d->B,
                                 d->dtype == LSTMSS_BF16, st);
    }));
    return LSTMSS_OK;
}

int64_t lstmss_bidir_workspace_bytes(const lstmss_dims *d, float sparsity,
                                     const lstmss_structure *s) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    Plan p;
    rc = make_plan(d, sparsity, s, s == nullptr || sparsity == 0.f, &p);
    if (rc)
        return rc;
    return (int64_t)bidir_layout(d, p).total;
}

int32_t lstm_bwd_bidir(const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                       const void *x, const void *x_rev, const void *W_fwd, const void *W_rev,
                       const void *cache_fwd, const void *cache_rev, const float *dH_up, float *dX,
                       float *dW_fwd, float *dW_rev, float *db_fwd, float *db_rev,
                       int32_t *idx_fwd, int32_t *idx_rev, void *ws, size_t ws_bytes,
                       void *stream) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    const bool dense = s == nullptr || sparsity == 0.f;
    Plan p;
    rc = make_plan(d, sparsity, s, dense, &p);
    if (rc)
        return rc;
    if (!x || !x_rev || !W_fwd || !W_rev || !cache_fwd || !cache_rev || !dH_up || !dW_fwd ||
        !dW_rev || !ws)
        return fail(LSTMSS_ERR_INVALID_ARG, "a required pointer is NULL");
    const BidirLayout Lb = bidir_layout(d, p);
    if (ws_bytes < Lb.total)
        return fail(LSTMSS_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", ws_bytes, Lb.total);
    StackRes *R = nullptr;
    HIP_TRY(stack_res(&R));
    std::unique_lock<std::mutex> lk(R->mu);
    return bidir_enqueue(d, dense, p, x, x_rev, W_fwd, W_rev, cache_fwd, cache_rev, dH_up, dX,
                         dW_fwd, dW_rev, db_fwd, db_rev, idx_fwd, idx_rev, ws, (hipStream_t)stream,
                         *R);
}

int64_t lstmss_stack_workspace_bytes(int32_t layers, const lstmss_dims *d, float sparsity,
                                     const lstmss_structure *s) {
    StackPlan sp;
    const int32_t rc = stack_plan(layers, d, sparsity, s, &sp);
    if (rc)
        return rc;
    return (int64_t)sp.total;
}

int32_t lstm_bwd_stack(int32_t layers, const lstmss_dims *d, float sparsity,
                       const lstmss_structure *s, const void *const *x, const void *const *W,
                       const void *const *cache, const float *dH_top, float *const *dX,
                       float *const *dW, float *const *db, int32_t *const *idx_out, void *ws,
                       size_t ws_bytes, void *stream) {
    StackPlan sp;
    int32_t rc = stack_plan(layers, d, sparsity, s, &sp);
    if (rc)
        return rc;
    if (!x || !W || !cache || !dH_top || !dX || !dW || !ws)
        return fail(LSTMSS_ERR_INVALID_ARG, "a required pointer is NULL");
    for (int l = 0; l < layers; ++l)
        if (!x[l] || !W[l] || !cache[l] || !dW[l] || (l > 0 && !dX[l]))
            return fail(LSTMSS_ERR_INVALID_ARG, "layer %d: a required pointer is NULL", l);
    if (ws_bytes < sp.total)
        return fail(LSTMSS_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", ws_bytes, sp.total);
    if (layers == 1)  // nothing to overlap: the single-layer call (graph-replayed)
        return backward(&d[0], sp.dense, sparsity, s, x[0], W[0], cache[0], dH_top, nullptr,
                        nullptr, dX[0], dW[0], db ? db[0] : nullptr, nullptr, nullptr,
                        idx_out ? idx_out[0] : nullptr, nullptr, ws, ws_bytes, stream);
    StackRes *R = nullptr;
    HIP_TRY(stack_res(&R));
    std::unique_lock<std::mutex> lk(R->mu);
    for (int l = 0; l < layers; ++l)  // one event per possible dX chunk
        while ((int)R->chunk_ev[l].size() < d[l].T) {
            hipEvent_t e = nullptr;
            HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
            R->chunk_ev[l].push_back(e);
        }
#if LSTMSS_STACK_GRAPHS
    // recorded into a HIP graph (built only for checking the capture against
    // a model of the stream-capture rules on the CPU)
    bool timing;
    {
        std::lock_guard<std::mutex> tl(g_tmu);
        timing = g_timing;
    }
    if (g_graphs && !timing) {
        auto u = [](const void *q) { return (uint64_t)(uintptr_t)q; };
        uint32_t spb;
        std::memcpy(&spb, &sparsity, 4);
        std::vector<uint64_t> key = {(uint64_t)layers, spb, u(dH_top), u(ws),
                                     (uint64_t)g_stack_dx_steps, (uint64_t)g_side_mode,
                                     s ? (uint64_t)s->kind : 99u, s ? (uint64_t)s->P : 0u,
                                     s ? (uint64_t)s->R : 0u, s ? (uint64_t)s->My : 0u,
                                     s ? (uint64_t)s->Mx : 0u};
        for (int l = 0; l < layers; ++l)
            for (uint64_t v : {(uint64_t)d[l].T, (uint64_t)d[l].B, (uint64_t)d[l].I,
                               (uint64_t)d[l].H, (uint64_t)d[l].dtype, u(x[l]), u(W[l]),
                               u(cache[l]), u(dX[l]), u(dW[l]), u(db ? db[l] : nullptr),
                               u(idx_out ? idx_out[l] : nullptr)})
                key.push_back(v);
        GraphEntry *hit = nullptr;
        for (GraphEntry &g : R->graphs)
            if (g.key == key)
                hit = &g;
        if (!hit) {
            HIP_TRY(hipStreamBeginCapture(R->cap, hipStreamCaptureModeRelaxed));
            rc = stack_enqueue(layers, d, sp, x, W, cache, dH_top, dX, dW, db, idx_out, ws, R->cap,
                               *R);
            hipGraph_t graph = nullptr;
            const hipError_t ec = hipStreamEndCapture(R->cap, &graph);
            if (rc != LSTMSS_OK) {
                if (graph)
                    (void)hipGraphDestroy(graph);
                return rc;
            }
            if (ec != hipSuccess)
                return fail(LSTMSS_ERR_HIP, "stack capture failed: %s", hipGetErrorString(ec));
            hipGraphExec_t exec = nullptr;
            const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
            (void)hipGraphDestroy(graph);
            if (ei != hipSuccess)
                return fail(LSTMSS_ERR_HIP, "stack graph instantiation failed: %s",
                            hipGetErrorString(ei));
            if (R->graphs.size() >= kMaxGraphs) {
                size_t oldest = 0;
                for (size_t i = 1; i < R->graphs.size(); ++i)
                    if (R->graphs[i].last_use < R->graphs[oldest].last_use)
                        oldest = i;
                (void)hipGraphExecDestroy(R->graphs[oldest].exec);
                R->graphs.erase(R->graphs.begin() + oldest);
            }
            R->graphs.push_back(GraphEntry{key, exec, 0});
            hit = &R->graphs.back();
        }
        hit->last_use = ++R->use_clock;
        HIP_TRY(hipGraphLaunch(hit->exec, (hipStream_t)stream));
        return LSTMSS_OK;
    }
#endif
    // enqueued directly on the layers' streams, whatever LSTMSS_OPT_GRAPHS
    // says: recording a stack call into a HIP graph ended in a host
    // segmentation fault on the GPU whose cause is not found (the capture
    // sequence satisfies the stream-capture rules as modelled on the CPU), so
    // that path is built only for the model
    return stack_enqueue(layers, d, sp, x, W, cache, dH_top, dX, dW, db, idx_out, ws,
                         (hipStream_t)stream, *R);
}

int32_t lstmss_version(void) { return LSTMSS_VERSION; }

const char *lstmss_strerror(int32_t code) {
    switch (code) {
    case LSTMSS_OK: return "success";
    case LSTMSS_ERR_INVALID_ARG: return "invalid argument";
    case LSTMSS_ERR_UNSUPPORTED: return "unsupported configuration";
    case LSTMSS_ERR_WORKSPACE: return "workspace too small";
    case LSTMSS_ERR_HIP: return "HIP runtime error";
    default: return "unknown error code";
    }
}

const char *lstmss_last_error(void) { return g_last_error.c_str(); }

int64_t lstmss_cache_bytes(const lstmss_dims *d) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    return (int64_t)cache_layout(d).total;
}

int64_t lstmss_kept_rows(const lstmss_dims *d, float sparsity, const lstmss_structure *s) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    Plan p;
    rc = make_plan(d, sparsity, s, false, &p);
    if (rc)
        return rc;
    return p.Kp;
}

int32_t lstmss_bwd_info(const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                        int32_t *flags) {
    if (!flags)
        return fail(LSTMSS_ERR_INVALID_ARG, "flags is NULL");
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    Plan p;
    rc = make_plan(d, sparsity, s, false, &p);
    if (rc)
        return rc;
    // a 256-byte aligned weight matrix and workspace
    const GatePath g = gate_path(d, p, false, (const void *)(uintptr_t)256,
                                 (const void *)(uintptr_t)256);
    *flags = (g.split ? LSTMSS_INFO_SPLIT_GATES : 0) |
             (g.select_in_product ? LSTMSS_INFO_SELECT_IN_PRODUCT : 0);
    return LSTMSS_OK;
}

int64_t lstmss_index_entries(const lstmss_dims *d, float sparsity, const lstmss_structure *s) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    Plan p;
    rc = make_plan(d, sparsity, s, false, &p);
    if (rc)
        return rc;
    return p.fine ? p.kept : p.Kp / p.P;
}

int64_t lstmss_workspace_bytes(const lstmss_dims *d, float sparsity, const lstmss_structure *s) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    Plan p;
    rc = make_plan(d, sparsity, s, s == nullptr || sparsity == 0.f, &p);
    if (rc)
        return rc;
    size_t total = ws_layout(d, p).total;
    if (s && sparsity == 0.f) {
        // lstm_bwd_structsparse at sparsity 0 runs its structure's plan (the
        // fine one indexes (4H / Mx) nb blocks and keeps block sums), which
        // may need more than the dense call
        Plan q;
        if (make_plan(d, sparsity, s, false, &q) == LSTMSS_OK)
            total = std::max(total, ws_layout(d, q).total);
    }
    return (int64_t)total;
}

// Forward workspace: the input projection of every step and the split-K
// partials of one step's recurrent product (both fp32).
struct FwdPlan {
    int splitk, tm, tn;
    long k_chunk;
    size_t zx, part, total;
};

FwdPlan fwd_plan(const lstmss_dims *d) {
    FwdPlan f;
    const bool bf16 = d->dtype == LSTMSS_BF16;
    const long G = 4L * d->H;
    gemm1_tile(bf16, d->B, G, 1, &f.tm, &f.tn);
    // enough work-groups for about three per CU in the recurrent product,
    // each split at least two 64-row stages long
    const long tiles = ceil_div(G, f.tm) * ceil_div(d->B, f.tn);
    const long want = ceil_div(768L, tiles);
    const long most = std::max(1L, (long)d->H / 128);
    long sk = std::max(1L, std::min(want, most));
    f.k_chunk = ceil_div(ceil_div((long)d->H, sk), GEMM1_TK) * GEMM1_TK;
    f.splitk = (int)ceil_div((long)d->H, f.k_chunk);
    const size_t GB = (size_t)G * d->B;
    f.zx = 0;
    f.part = align256((size_t)d->T * GB * 4);
    f.total = f.part + align256((size_t)f.splitk * GB * 4);
    return f;
}

int64_t lstmss_fwd_workspace_bytes(const lstmss_dims *d) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    return (int64_t)fwd_plan(d).total;
}

int32_t lstm_fwd_cache(const lstmss_dims *d, const void *x, const void *W, const float *b,
                       const float *h0, const float *c0, void *h_out, void *cache, void *ws,
                       size_t ws_bytes, void *stream) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    if (!x || !W || !cache)
        return fail(LSTMSS_ERR_INVALID_ARG, "a required pointer is NULL");
    const FwdPlan F = fwd_plan(d);
    if (ws && ws_bytes < F.total)
        return fail(LSTMSS_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", ws_bytes, F.total);
    hipStream_t st = (hipStream_t)stream;
    const bool bf16 = d->dtype == LSTMSS_BF16;
    const size_t es = elem_bytes(d->dtype);
    const long HB = (long)d->H * d->B, G = 4L * d->H, K = (long)d->I + d->H;
    const CacheLayout C = cache_layout(d);
    char *cb = (char *)cache;
    float *cst = (float *)(cb + C.c);
    char *hst = cb + C.h;
    HIP_TRY(launch_copy_in(cst, c0, HB, st));
    HIP_TRY(launch_h0_store(hst, h0, HB, bf16, st));
    if (!ws) {
        // no scratch: one fused product + cell-update kernel per step
        for (int t = 0; t < d->T; ++t) {
            FwdArgs f{};
            f.W = W; f.bias = b;
            f.xt = (const char *)x + (size_t)t * d->I * d->B * es;
            f.hp = hst + (size_t)t * HB * es;
            f.cp = cst + (size_t)t * HB;
            f.I = d->I; f.H = d->H; f.B = d->B;
            f.gates = cb + C.gates + (size_t)t * G * d->B * es;
            f.cn = cst + (size_t)(t + 1) * HB;
            f.hn = hst + (size_t)(t + 1) * HB * es;
            f.hout = h_out ? (char *)h_out + (size_t)t * HB * es : nullptr;
            HIP_TRY(timed(LSTMSS_KERNEL_FORWARD, st, [&] { return launch_fwd_step(f, bf16, st); }));
        }
        return LSTMSS_OK;
    }
    char *wb = (char *)ws;
    float *zx = (float *)(wb + F.zx);
    float *part = (float *)(wb + F.part);
    // input projection W_x x_t of every step in one launch (steps batched)
    Gemm1Args gi{};
    gi.W = W; gi.ldw = K; gi.kcol0 = 0; gi.Gc = x; gi.Kp = d->I; gi.M = (int)G; gi.m_begin = 0;
    gi.N = d->B; gi.out_row0 = 0; gi.part = zx; gi.part_stride = 0; gi.splitk = 1;
    gi.k_chunk = ceil_div((long)d->I, GEMM1_TK) * GEMM1_TK; gi.steps = d->T;
    gi.gc_step = (long)d->I * d->B; gi.out_step = G * d->B;
    gi.dma = g_gemm_dma ? 1 : 0;
    HIP_TRY(timed(LSTMSS_KERNEL_FORWARD, st, [&] { return launch_gemm_fwd(gi, bf16, st); }));
    for (int t = 0; t < d->T; ++t) {
        // recurrent product W_h h_{t-1}, split over k
        Gemm1Args gr{};
        gr.W = W; gr.ldw = K; gr.kcol0 = d->I; gr.Gc = hst + (size_t)t * HB * es; gr.Kp = d->H;
        gr.M = (int)G; gr.m_begin = 0; gr.N = d->B; gr.out_row0 = 0; gr.part = part;
        gr.part_stride = G * d->B; gr.splitk = F.splitk; gr.k_chunk = F.k_chunk; gr.steps = 1;
        gr.tm = F.tm; gr.tn = F.tn; gr.dma = g_gemm_dma ? 1 : 0;
        HIP_TRY(timed(LSTMSS_KERNEL_FORWARD, st, [&] { return launch_gemm_fwd(gr, bf16, st); }));
        FwdActArgs fa{};
        fa.zx = zx + (size_t)t * G * d->B;
        fa.part = part; fa.nparts = F.splitk; fa.part_stride = G * d->B;
        fa.bias = b; fa.cp = cst + (size_t)t * HB; fa.H = d->H; fa.B = d->B;
        fa.gates = cb + C.gates + (size_t)t * G * d->B * es;
        fa.cn = cst + (size_t)(t + 1) * HB;
        fa.hn = hst + (size_t)(t + 1) * HB * es;
        fa.hout = h_out ? (char *)h_out + (size_t)t * HB * es : nullptr;
        HIP_TRY(timed(LSTMSS_KERNEL_FORWARD, st, [&] { return launch_fwd_act(fa, bf16, st); }));
    }
    return LSTMSS_OK;
}

int32_t lstmss_sgd_update(const lstmss_dims *d, void *W, float *b, const float *dW,
                          const float *db, float lr, void *stream) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    if (!W || !dW || (b && !db))
        return fail(LSTMSS_ERR_INVALID_ARG, "a required pointer is NULL");
    if (!std::isfinite(lr))
        return fail(LSTMSS_ERR_INVALID_ARG, "learning rate %g is not finite", (double)lr);
    const long G = 4L * d->H;
    hipStream_t st = (hipStream_t)stream;
    HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] {
        return launch_sgd(W, dW, G * ((long)d->I + d->H), b, db, b ? G : 0, lr,
                          d->dtype == LSTMSS_BF16, st);
    }));
    return LSTMSS_OK;
}

int32_t lstmss_mse_grad(const lstmss_dims *d, const void *h, const float *y, float *dH,
                        double *loss, void *stream) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    if (!h || !y || !dH)
        return fail(LSTMSS_ERR_INVALID_ARG, "a required pointer is NULL");
    const long n = (long)d->T * d->H * d->B;
    hipStream_t st = (hipStream_t)stream;
    HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] {
        return launch_mse(h, y, dH, n, 1.f / (float)d->B, loss, LSTMSS_LOSS_SLOTS - 1,
                          d->dtype == LSTMSS_BF16, st);
    }));
    return LSTMSS_OK;
}

int32_t lstm_bwd_dense(const lstmss_dims *d, const void *x, const void *W, const void *cache,
                       const float *dH_up, const float *dhT, const float *dcT, float *dX,
                       float *dW, float *db, float *dh0, float *dc0, void *ws, size_t ws_bytes,
                       void *stream) {
    return backward(d, true, 0.f, nullptr, x, W, cache, dH_up, dhT, dcT, dX, dW, db, dh0, dc0,
                    nullptr, nullptr, ws, ws_bytes, stream);
}

int32_t lstm_bwd_structsparse(const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                              const void *x, const void *W, const void *cache,
                              const float *dH_up, const float *dhT, const float *dcT, float *dX,
                              float *dW, float *db, float *dh0, float *dc0, int32_t *idx_out,
                              void *dbg_dgates, void *ws, size_t ws_bytes, void *stream) {
    return backward(d, false, sparsity, s, x, W, cache, dH_up, dhT, dcT, dX, dW, db, dh0, dc0,
                    idx_out, dbg_dgates, ws, ws_bytes, stream);
}

int64_t lstmss_select_workspace_bytes(const lstmss_dims *d, float sparsity,
                                      const lstmss_structure *s) {
    return lstmss::select_scratch_bytes(d, sparsity, s);
}

int32_t lstmss_select_compact(const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                              const void *dG, void *dG_c, int32_t *idx, double *scores, void *ws,
                              size_t ws_bytes, void *stream) {
    return lstmss::select_compact_impl(d, sparsity, s, dG, dG_c, idx, scores, ws, ws_bytes, stream,
                                       true);
}

int32_t lstmss_set_option(int32_t option, int32_t value) {
    std::lock_guard<std::mutex> lk(g_side_mu);
    for (auto &kv : g_side) {  // graphs recorded under the old setting are dropped
        std::lock_guard<std::mutex> l2(kv.second.mu);
        for (GraphEntry &g : kv.second.graphs)
            (void)hipGraphExecDestroy(g.exec);
        kv.second.graphs.clear();
    }
#if LSTMSS_STACK_GRAPHS
    for (auto &kv : g_stack) {
        std::lock_guard<std::mutex> l2(kv.second.mu);
        for (GraphEntry &g : kv.second.graphs)
            (void)hipGraphExecDestroy(g.exec);
        kv.second.graphs.clear();
    }
#endif
    switch (option) {
    case LSTMSS_OPT_GRAPHS: g_graphs = value != 0; return LSTMSS_OK;
    case LSTMSS_OPT_FINE_SKIP: g_fine_skip = value != 0; return LSTMSS_OK;
    case LSTMSS_OPT_GEMM_DMA: g_gemm_dma = value != 0; return LSTMSS_OK;
    case LSTMSS_OPT_GEMM_SELECT: g_gemm_select = value != 0; return LSTMSS_OK;
    case LSTMSS_OPT_FINE_FUSED: g_fine_fused = value != 0; return LSTMSS_OK;
    case LSTMSS_OPT_WGRAD_BIG: g_wgrad_big = value != 0; return LSTMSS_OK;
    case LSTMSS_OPT_STACK_DX_STEPS:
        if (value < 0)
            return fail(LSTMSS_ERR_INVALID_ARG, "stack dX steps %d must be >= 0", value);
        g_stack_dx_steps = value;
        return LSTMSS_OK;
    case LSTMSS_OPT_SIDE_STREAM:
        if (value < 0 || value > 2)
            return fail(LSTMSS_ERR_INVALID_ARG, "side-stream mode %d (0, 1 or 2)", value);
        g_side_mode = value;
        return LSTMSS_OK;
    default: return fail(LSTMSS_ERR_INVALID_ARG, "unknown option %d", option);
    }
}

int32_t lstmss_timing_enable(int32_t on) {
    std::lock_guard<std::mutex> lk(g_tmu);
    g_timing = on != 0;
    return LSTMSS_OK;
}

int32_t lstmss_timing_read(int32_t kind, double *total_ms, int64_t *launches) {
    if (kind < 0 || kind >= LSTMSS_KERNEL_KINDS || !total_ms || !launches)
        return fail(LSTMSS_ERR_INVALID_ARG, "bad timing query");
    std::lock_guard<std::mutex> lk(g_tmu);
    for (const TimingRec &r : g_pending) {
        float ms = 0.f;
        HIP_TRY(hipEventSynchronize(r.b));
        HIP_TRY(hipEventElapsedTime(&ms, r.a, r.b));
        g_total_ms[r.kind] += ms;
        g_count[r.kind] += 1;
        g_event_pool.push_back(r.a);
        g_event_pool.push_back(r.b);
    }
    g_pending.clear();
    *total_ms = g_total_ms[kind];
    *launches = g_count[kind];
    return LSTMSS_OK;
}

int32_t lstmss_timing_reset(void) {
    std::lock_guard<std::mutex> lk(g_tmu);
    for (const TimingRec &r : g_pending) {
        (void)hipEventSynchronize(r.b);
        g_event_pool.push_back(r.a);
        g_event_pool.push_back(r.b);
    }
    g_pending.clear();
    for (int k = 0; k < LSTMSS_KERNEL_KINDS; ++k) {
        g_total_ms[k] = 0.0;
        g_count[k] = 0;
    }
    return LSTMSS_OK;
}

} // extern "C"
