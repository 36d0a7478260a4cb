// Drives the library's host code, built against the stream-capture model, through
// the call sequences the GPU tests make: stack calls recorded into graphs and
// replayed, re-recorded with other arguments (events reused across captures),
// single-layer calls recorded in between, direct calls after recorded ones,
// the side-stream mode, bidirectional calls on the same streams; coarse,
// fine and dense, fp32 and bf16, small shapes and the two-kernel gate path.
// Prints every violation of the modelled rules; exit status 1 if any.
#include "../../include/lstmss.h"

#include "hip/hip_runtime.h"

#include <cstdint>
#include <cstdio>
#include <string>
#include <vector>

extern "C" {
int hipsim_violation_count();
const char *hipsim_violation(int i);
long hipsim_launches();
long hipsim_captured_nodes();
int hipsim_captures();
int hipsim_streams_capturing();
int hipsim_enqueue(hipStream_t s, const char *what);
}

namespace {

// distinct, 256-byte aligned stand-in device addresses (never dereferenced)
uintptr_t g_next = 1 << 20;
void *fake(size_t bytes) {
    void *p = (void *)g_next;
    g_next += (bytes + 4095) & ~(size_t)4095;
    return p;
}

int g_fail = 0;

void check(int32_t rc, const char *what) {
    if (rc != LSTMSS_OK) {
        std::printf("call failed: %s: %d %s\n", what, rc, lstmss_last_error());
        g_fail = 1;
    }
}

struct Stack {
    int layers;
    std::vector<lstmss_dims> d;
    std::vector<const void *> x, W, cache;
    std::vector<float *> dX, dW, db;
    std::vector<int32_t *> idx;
    const float *dH;
    void *ws;
    size_t ws_bytes;
};

Stack make_stack(int layers, int T, int B, int I, int H, int dtype, float sp,
                 const lstmss_structure *s) {
    Stack k;
    k.layers = layers;
    for (int l = 0; l < layers; ++l) {
        lstmss_dims d{T, B, l == 0 ? I : H, H, dtype};
        k.d.push_back(d);
        const size_t es = dtype == LSTMSS_BF16 ? 2 : 4;
        k.x.push_back(fake((size_t)T * d.I * B * es));
        k.W.push_back(fake((size_t)4 * H * (d.I + H) * es));
        k.cache.push_back(fake((size_t)lstmss_cache_bytes(&d)));
        k.dX.push_back((float *)fake((size_t)T * d.I * B * 4));
        k.dW.push_back((float *)fake((size_t)4 * H * (d.I + H) * 4));
        k.db.push_back((float *)fake((size_t)4 * H * 4));
        k.idx.push_back(s ? (int32_t *)fake((size_t)T * lstmss_index_entries(&d, sp, s) * 4)
                          : nullptr);
    }
    k.dH = (const float *)fake((size_t)T * H * B * 4);
    const int64_t n = lstmss_stack_workspace_bytes(layers, k.d.data(), sp, s);
    if (n < 0) {
        std::printf("workspace query failed: %lld\n", (long long)n);
        g_fail = 1;
    }
    k.ws_bytes = (size_t)(n > 0 ? n : 0);
    k.ws = fake(k.ws_bytes);
    return k;
}

void run_stack(const Stack &k, float sp, const lstmss_structure *s, const char *what) {
    check(lstm_bwd_stack(k.layers, k.d.data(), sp, s, k.x.data(), k.W.data(), k.cache.data(), k.dH,
                         k.dX.data(), k.dW.data(), k.db.data(), s ? k.idx.data() : nullptr, k.ws,
                         k.ws_bytes, nullptr),
          what);
}

void run_layer(const Stack &k, int l, float sp, const lstmss_structure *s, const char *what) {
    const int64_t n = lstmss_workspace_bytes(&k.d[l], sp, s);
    void *ws = fake((size_t)n);
    if (s)
        check(lstm_bwd_structsparse(&k.d[l], sp, s, k.x[l], k.W[l], k.cache[l], k.dH, nullptr,
                                    nullptr, k.dX[l], k.dW[l], k.db[l], nullptr, nullptr, k.idx[l],
                                    nullptr, ws, (size_t)n, nullptr),
              what);
    else
        check(lstm_bwd_dense(&k.d[l], k.x[l], k.W[l], k.cache[l], k.dH, nullptr, nullptr, k.dX[l],
                             k.dW[l], k.db[l], nullptr, nullptr, ws, (size_t)n, nullptr),
              what);
}

void run_bidir(int T, int B, int I, int H, float sp, const lstmss_structure *s) {
    lstmss_dims d{T, B, I, H, LSTMSS_F32};
    const int64_t n = lstmss_bidir_workspace_bytes(&d, sp, s);
    void *ws = fake((size_t)n);
    check(lstm_bwd_bidir(&d, sp, s, fake(T * I * B * 4), fake(T * I * B * 4), fake(4 * H * (I + H) * 4),
                         fake(4 * H * (I + H) * 4), fake(lstmss_cache_bytes(&d)),
                         fake(lstmss_cache_bytes(&d)), (const float *)fake(T * 2 * H * B * 4),
                         (float *)fake(T * I * B * 4), (float *)fake(4 * H * (I + H) * 4),
                         (float *)fake(4 * H * (I + H) * 4), (float *)fake(4 * H * 4),
                         (float *)fake(4 * H * 4), nullptr, nullptr, ws, (size_t)n, nullptr),
          "bidir");
}

} // namespace

// The model must flag each forbidden sequence (planted here, on the CPU).
int selftest() {
    int bad = 0;
    auto expect = [&](const char *what, int before) {
        const bool seen = hipsim_violation_count() > before;
        std::printf("%s: %s\n", what, seen ? "flagged" : "NOT FLAGGED");
        bad += !seen;
    };
    hipStream_t s1, s2, s3;
    hipEvent_t e1, e2;
    hipGraph_t g = nullptr;
    hipStreamCreateWithFlags(&s1, hipStreamNonBlocking);
    hipStreamCreateWithFlags(&s2, hipStreamNonBlocking);
    hipStreamCreateWithFlags(&s3, hipStreamNonBlocking);
    hipEventCreateWithFlags(&e1, hipEventDisableTiming);
    hipEventCreateWithFlags(&e2, hipEventDisableTiming);
    int n = hipsim_violation_count();
    hipStreamBeginCapture(nullptr, hipStreamCaptureModeRelaxed);
    expect("capture on the null stream", n);
    // a forked stream that never joins back
    n = hipsim_violation_count();
    hipStreamBeginCapture(s1, hipStreamCaptureModeRelaxed);
    hipEventRecord(e1, s1);
    hipStreamWaitEvent(s2, e1, 0);
    hipsim_enqueue(s2, "work");
    hipStreamEndCapture(s1, &g);
    expect("unjoined stream", n);
    // a wait on an event of the ended capture
    n = hipsim_violation_count();
    hipStreamWaitEvent(s3, e1, 0);
    expect("wait on an event of an ended capture", n);
    // two captures merged by a wait
    n = hipsim_violation_count();
    hipStreamBeginCapture(s1, hipStreamCaptureModeRelaxed);
    hipStreamBeginCapture(s2, hipStreamCaptureModeRelaxed);
    hipEventRecord(e2, s2);
    hipStreamWaitEvent(s1, e2, 0);
    expect("merge of two captures", n);
    hipStreamEndCapture(s2, &g);
    // a capturing stream waiting on work recorded outside the capture
    n = hipsim_violation_count();
    hipEventRecord(e2, s3);
    hipStreamWaitEvent(s1, e2, 0);
    expect("wait on an event recorded outside the capture", n);
    // a synchronisation on a captured event
    n = hipsim_violation_count();
    hipEventRecord(e1, s1);
    hipEventSynchronize(e1);
    expect("synchronize on a captured event", n);
    hipStreamEndCapture(s1, &g);
    // a capture ended on a stream that is not its origin
    n = hipsim_violation_count();
    hipStreamBeginCapture(s1, hipStreamCaptureModeRelaxed);
    hipStreamEndCapture(s2, &g);
    expect("end capture on a stream that is not the origin", n);
    hipStreamEndCapture(s1, &g);
    return bad;
}

int main(int argc, char **argv) {
    if (argc > 1 && std::string(argv[1]) == "--selftest") {
        const int bad = selftest();
        std::printf("selftest: %d forbidden sequences not flagged\n", bad);
        return bad ? 1 : 0;
    }
    const lstmss_structure coarse{LSTMSS_COARSE, 4, 8, 0, 0};
    const lstmss_structure fine{LSTMSS_FINE, 0, 0, 16, 4};
    const lstmss_structure fine32{LSTMSS_FINE, 0, 0, 32, 32};

    // the two-kernel gate path with the selection inside the dh product
    Stack a = make_stack(2, 26, 128, 2048, 2048, LSTMSS_F32, 0.5f, &coarse);
    run_stack(a, 0.5f, &coarse, "stack capture");
    run_stack(a, 0.5f, &coarse, "stack replay");
    // other arguments: a new capture reusing the same streams and events
    Stack b = make_stack(3, 12, 64, 96, 128, LSTMSS_F32, 0.5f, &coarse);
    run_stack(b, 0.5f, &coarse, "stack capture, small shape");
    run_layer(b, 1, 0.5f, &coarse, "single-layer capture in between");
    run_stack(b, 0.5f, &coarse, "stack replay after a single-layer capture");
    run_stack(a, 0.5f, &coarse, "first stack replayed again");
    // dense, fine, bf16, a ragged last dX chunk
    Stack c = make_stack(2, 8, 128, 64, 64, LSTMSS_F32, 0.f, nullptr);
    run_stack(c, 0.f, nullptr, "dense stack capture");
    Stack f = make_stack(2, 7, 64, 32, 64, LSTMSS_F32, 0.5f, &fine);
    run_stack(f, 0.5f, &fine, "fine stack capture");
    Stack f32 = make_stack(3, 10, 64, 64, 64, LSTMSS_F32, 0.5f, &fine32);
    run_stack(f32, 0.5f, &fine32, "fine 32x32 stack capture");
    Stack h = make_stack(2, 6, 64, 64, 128, LSTMSS_BF16, 0.5f, &coarse);
    run_stack(h, 0.5f, &coarse, "bf16 stack capture");
    lstmss_set_option(2, 5);  // five steps per dX launch: ragged chunks
    run_stack(b, 0.5f, &coarse, "stack capture, 5-step dX chunks");
    lstmss_set_option(2, 0);
    // the side stream in every layer (fork ring and join events in the capture)
    lstmss_set_option(1, 1);
    run_stack(b, 0.5f, &coarse, "stack capture with side streams");
    run_stack(b, 0.5f, &coarse, "stack replay with side streams");
    run_layer(b, 0, 0.5f, &coarse, "single-layer capture with a side stream");
    lstmss_set_option(1, 2);
    // bidirectional calls on the same per-device streams and events
    run_bidir(10, 64, 48, 96, 0.5f, &coarse);
    run_stack(a, 0.5f, &coarse, "stack capture after a bidirectional call");
    // direct calls after recorded ones (events last recorded in a capture)
    lstmss_set_option(0, 0);
    run_stack(a, 0.5f, &coarse, "direct stack call");
    run_layer(a, 0, 0.5f, &coarse, "direct single-layer call");
    run_bidir(10, 64, 48, 96, 0.5f, &coarse);
    lstmss_set_option(0, 1);
    run_stack(b, 0.5f, &coarse, "stack capture after direct calls");

    const int nv = hipsim_violation_count();
    std::printf("launches %ld, captured nodes %ld, captures %d, streams left capturing %d, "
                "violations %d\n",
                hipsim_launches(), hipsim_captured_nodes(), hipsim_captures(),
                hipsim_streams_capturing(), nv);
    for (int i = 0; i < nv && i < 50; ++i)
        std::printf("violation: %s\n", hipsim_violation(i));
    return (nv || g_fail || hipsim_streams_capturing()) ? 1 : 0;
}
