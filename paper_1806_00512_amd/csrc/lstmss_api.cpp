// Host side of liblstmss: argument checks, cache / workspace layout and the
// backward-through-time driver (one layer per call, reverse time loop).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
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

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
long ceil_div(long a, long b) { return (a + b - 1) / b; }

// LDS budget of the fused gate-gradient / selection kernel's work-group.
constexpr size_t kMaxLds = 64 * 1024;
// Largest K range one data-gradient work-group covers (its LDS row table).
constexpr long kGemm1KcMax = 4096;

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
    long kept;     // kept slices per step
    long Kp;       // kept rows per step
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
    if (s->kind == LSTMSS_FINE)
        return fail(LSTMSS_ERR_UNSUPPORTED, "fine-grained structure is not built");
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

int splitk_for(const lstmss_dims *d, long Kp) {
    const long M = (long)d->I + d->H;
    const long tiles = ceil_div(M, gemm1_tm(d->B)) * ceil_div(d->B, gemm1_tn(d->B));
    long sk = ceil_div(512, tiles);
    const long max_sk = std::max(1L, Kp / (4L * GEMM1_TK));
    sk = std::min(std::max(sk, 1L), max_sk);
    return (int)std::min(sk, 64L);
}

struct WsLayout {
    size_t dc0, dc1, part, dGc, idx, db, total;
    int splitk;
    long k_chunk;
};

WsLayout ws_layout(const lstmss_dims *d, const Plan &p) {
    const size_t es = elem_bytes(d->dtype);
    const size_t HB = (size_t)d->H * d->B;
    WsLayout L;
    L.splitk = std::max<int>(splitk_for(d, p.Kp), (int)ceil_div(p.Kp, kGemm1KcMax));
    L.k_chunk = ceil_div(ceil_div(p.Kp, L.splitk), GEMM1_TK) * GEMM1_TK;
    L.splitk = (int)ceil_div(p.Kp, L.k_chunk);
    size_t off = 0;
    L.dc0 = off; off += align256(HB * 4);
    L.dc1 = off; off += align256(HB * 4);
    L.part = off; off += align256((size_t)L.splitk * ((size_t)d->I + d->H) * d->B * 4);
    L.dGc = off; off += align256((size_t)d->T * p.Kp * d->B * es);
    L.idx = off; off += align256((size_t)d->T * p.kept * 4);
    L.db = off; off += align256((size_t)4 * d->H * 4);
    L.total = off;
    return L;
}

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
    const bool bf16 = d->dtype == LSTMSS_BF16;
    const bool sparse = !dense;
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

    // weight gradient: one batched launch after the time loop when the
    // structure fits its routing tiles, else a per-step accumulation
    const bool batched = !sparse || wgrad_supported(p.P, p.R, p.S);
    if (!batched)
        HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] { return launch_fill(dW, G * K, 0.f, st); }));
    HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] { return launch_fill(dbp, G, 0.f, st); }));

    const long part_stride = K * B;
    const int m_begin = dX ? 0 : I;
    for (int t = T - 1; t >= 0; --t) {
        const bool last = t == T - 1;
        char *dGc = dGc_all + (size_t)t * p.Kp * B * es;
        int32_t *idx = idx_all + (size_t)t * p.kept;

        CellArgs ca{};
        ca.B = B; ca.H = H; ca.I = I;
        ca.P = sparse ? p.P : 1; ca.R = sparse ? p.R : 1; ca.S = sparse ? p.S : 0;
        ca.nslices = sparse ? p.nslices : G;
        ca.regions_per_wg = 1;
        if (sparse) {
            const int rows_per_region = p.R * p.P;
            ca.regions_per_wg = std::max(1, 32 / rows_per_region);
        } else {
            ca.regions_per_wg = 32;  // dense: 32 rows per work-group
        }
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
            ca.dh_part = part + (size_t)I * B;
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
        if (!last && dX) {
            ca.dx_part = part;
            ca.dx_nparts = L.splitk;
            ca.dx_stride = part_stride;
            ca.dx_out = dX + (size_t)(t + 1) * I * B;
            ca.dx_n = (long)I * B;
        }
        if (cell_lds_bytes(ca, sparse ? CELL_SPARSE : CELL_DENSE) > kMaxLds)
            return fail(LSTMSS_ERR_UNSUPPORTED, "R*P*B too large for one work-group's LDS");
        HIP_TRY(timed(LSTMSS_KERNEL_GATES, st, [&] { return launch_cell(ca, sparse ? CELL_SPARSE : CELL_DENSE, bf16, st); }));

        Gemm1Args g1{};
        g1.W = W; g1.ldw = K; g1.Gc = dGc; g1.idx = sparse ? idx : nullptr; g1.P = p.P;
        g1.Kp = p.Kp; g1.M = (int)K; g1.m_begin = m_begin; g1.N = B;
        g1.part = part; g1.part_stride = part_stride; g1.splitk = L.splitk; g1.k_chunk = L.k_chunk;
        HIP_TRY(timed(LSTMSS_KERNEL_DATA_GRAD, st, [&] { return launch_gemm1(g1, bf16, st); }));

        if (!batched) {
            Gemm2Args g2{};
            g2.Gc = dGc; g2.idx = sparse ? idx : nullptr; g2.P = p.P; g2.Kp = p.Kp;
            g2.xt = (const char *)x + (size_t)t * I * B * es;
            g2.hp = hst + (size_t)t * HB * es;
            g2.I = I; g2.H = H; g2.B = B; g2.dW = dW;
            HIP_TRY(timed(LSTMSS_KERNEL_WEIGHT_GRAD, st, [&] { return launch_gemm2(g2, bf16, st); }));
        }
    }
    if (batched) {
        WgradArgs wg{};
        wg.Gc = dGc_all; wg.idx = sparse ? idx_all : nullptr; wg.x = x; wg.h = hst;
        wg.T = T; wg.I = I; wg.H = H; wg.B = B; wg.Kp = (int)p.Kp; wg.kept = (int)p.kept;
        wg.P = p.P; wg.R = p.R; wg.S = p.S; wg.dW = dW;
        HIP_TRY(timed(LSTMSS_KERNEL_WEIGHT_GRAD, st, [&] { return launch_wgrad(wg, sparse, bf16, st); }));
    }
    if (dX)
        HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] { return launch_reduce_parts(dX, part, L.splitk, part_stride, (long)I * B, st); }));
    if (dh0)
        HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] { return launch_reduce_parts(dh0, part + (size_t)I * B, L.splitk, part_stride, HB, st); }));
    if (dc0)
        HIP_TRY(timed(LSTMSS_KERNEL_AUX, st, [&] { return launch_copy_in(dc0, dcbuf[0], HB, st); }));
    return LSTMSS_OK;
}

} // namespace

extern "C" {

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

int64_t lstmss_workspace_bytes(const lstmss_dims *d, float sparsity, const lstmss_structure *s) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    Plan p;
    rc = make_plan(d, sparsity, s, s == nullptr || sparsity == 0.f, &p);
    if (rc)
        return rc;
    return (int64_t)ws_layout(d, p).total;
}

int32_t lstm_fwd_cache(const lstmss_dims *d, const void *x, const void *W, const float *b,
                       const float *h0, const float *c0, void *h_out, void *cache,
                       void *stream) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    if (!x || !W || !cache)
        return fail(LSTMSS_ERR_INVALID_ARG, "a required pointer is NULL");
    hipStream_t st = (hipStream_t)stream;
    const bool bf16 = d->dtype == LSTMSS_BF16;
    const size_t es = elem_bytes(d->dtype);
    const long HB = (long)d->H * d->B, G = 4L * d->H;
    const CacheLayout C = cache_layout(d);
    char *cb = (char *)cache;
    float *cst = (float *)(cb + C.c);
    char *hst = cb + C.h;
    HIP_TRY(launch_copy_in(cst, c0, HB, st));
    HIP_TRY(launch_h0_store(hst, h0, HB, bf16, st));
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

int32_t lstmss_select_compact(const lstmss_dims *d, float sparsity, const lstmss_structure *s,
                              const void *dG, void *dG_c, int32_t *idx, double *scores,
                              void *stream) {
    int32_t rc = check_dims(d);
    if (rc)
        return rc;
    Plan p;
    rc = make_plan(d, sparsity, s, false, &p);
    if (rc)
        return rc;
    if (!dG || !dG_c || !idx)
        return fail(LSTMSS_ERR_INVALID_ARG, "a required pointer is NULL");
    CellArgs ca{};
    ca.B = d->B; ca.H = d->H; ca.I = d->I;
    ca.P = p.P; ca.R = p.R; ca.S = p.S;
    ca.nslices = p.nslices;
    ca.regions_per_wg = std::max(1, 32 / (p.R * p.P));
    ca.dG_in = dG;
    ca.dGc = dG_c;
    ca.idx = idx;
    ca.scores = scores;
    if (cell_lds_bytes(ca, CELL_GIVEN) > kMaxLds)
        return fail(LSTMSS_ERR_UNSUPPORTED, "R*P*B too large for one work-group's LDS");
    hipStream_t st = (hipStream_t)stream;
    HIP_TRY(timed(LSTMSS_KERNEL_GATES, st, [&] { return launch_cell(ca, CELL_GIVEN, d->dtype == LSTMSS_BF16, st); }));
    return LSTMSS_OK;
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
