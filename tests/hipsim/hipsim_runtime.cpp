// A model of the HIP stream / event / stream-capture semantics the library's
// host driver relies on, for checking its capture paths on the CPU.  Streams
// carry the capture they belong to and their last captured nodes; events
// carry the capture and nodes they were last recorded at; a capture ends
// only when every stream that joined it has joined back into the origin.
// Whatever the documented rules forbid (a wait that would merge two captures
// or isolate one, a wait on an event of an ended or destroyed capture, a
// launch into an ended capture, an unjoined stream, a synchronisation on a
// captured event, capture on the null stream) is recorded as a violation
// instead of crashing, so that a driver run lists them all.
#include "hip/hip_runtime.h"

#include <cstdarg>
#include <cstdio>
#include <memory>
#include <set>
#include <string>
#include <vector>

namespace {

struct Capture;

struct Node {
    int id;
    std::vector<Node *> deps;
    std::string what;
};

struct Capture {
    int id;
    ihipStream_t *origin;
    enum { ACTIVE, ENDED, INVALID } status = ACTIVE;
    std::vector<std::unique_ptr<Node>> nodes;
    std::set<ihipStream_t *> joined;
    bool graph_destroyed = false;
};

std::vector<std::unique_ptr<Capture>> g_captures;
std::vector<std::string> g_violations;
int g_next_id = 1;
long g_launches = 0, g_captured_nodes = 0;

void violation(const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_violations.push_back(buf);
}

} // namespace

struct ihipStream_t {
    int id;
    unsigned flags;
    Capture *cap = nullptr;
    std::vector<Node *> deps;  // last nodes of this stream inside its capture
};

struct ihipEvent_t {
    int id;
    Capture *cap = nullptr;  // capture it was last recorded in, or null
    std::vector<Node *> deps;
    bool recorded = false;
};

struct ihipGraph {
    Capture *cap;
    bool destroyed = false;
};

struct hipGraphExec {
    ihipGraph *graph;
    long nodes;
};

namespace {

std::vector<std::unique_ptr<ihipStream_t>> g_streams;
std::vector<std::unique_ptr<ihipEvent_t>> g_events;
std::vector<std::unique_ptr<ihipGraph>> g_graphs;
std::vector<std::unique_ptr<hipGraphExec>> g_execs;

// every node reachable backwards from `from`
void ancestors(const std::vector<Node *> &from, std::set<Node *> *out) {
    std::vector<Node *> todo(from.begin(), from.end());
    while (!todo.empty()) {
        Node *n = todo.back();
        todo.pop_back();
        if (!out->insert(n).second)
            continue;
        for (Node *d : n->deps)
            todo.push_back(d);
    }
}

} // namespace

extern "C" {

// adds a kernel (or other work item) to stream s; called by the stub launchers
int hipsim_enqueue(hipStream_t s, const char *what) {
    ++g_launches;
    if (!s)
        return hipSuccess;  // the null stream: never captured by the library
    if (!s->cap)
        return hipSuccess;
    Capture *c = s->cap;
    if (c->status != Capture::ACTIVE) {
        violation("launch of %s into capture %d, which is %s", what, c->id,
                  c->status == Capture::ENDED ? "ended" : "invalidated");
        return hipErrorStreamCaptureInvalidated;
    }
    auto n = std::make_unique<Node>();
    n->id = g_next_id++;
    n->deps = s->deps;
    n->what = what;
    s->deps = {n.get()};
    c->nodes.push_back(std::move(n));
    ++g_captured_nodes;
    return hipSuccess;
}

int hipsim_violation_count() { return (int)g_violations.size(); }
const char *hipsim_violation(int i) { return g_violations.at(i).c_str(); }
long hipsim_launches() { return g_launches; }
long hipsim_captured_nodes() { return g_captured_nodes; }
int hipsim_captures() { return (int)g_captures.size(); }
int hipsim_streams_capturing() {
    int n = 0;
    for (auto &s : g_streams)
        n += s->cap != nullptr;
    return n;
}

} // extern "C"

hipError_t hipGetDevice(int *dev) {
    *dev = 0;
    return hipSuccess;
}

hipError_t hipDeviceGetAttribute(int *v, hipDeviceAttribute_t, int) {
    *v = 256;
    return hipSuccess;
}

hipError_t hipStreamCreateWithFlags(hipStream_t *s, unsigned flags) {
    auto p = std::make_unique<ihipStream_t>();
    p->id = g_next_id++;
    p->flags = flags;
    *s = p.get();
    g_streams.push_back(std::move(p));
    return hipSuccess;
}

hipError_t hipEventCreateWithFlags(hipEvent_t *e, unsigned) {
    auto p = std::make_unique<ihipEvent_t>();
    p->id = g_next_id++;
    *e = p.get();
    g_events.push_back(std::move(p));
    return hipSuccess;
}

hipError_t hipEventCreate(hipEvent_t *e) { return hipEventCreateWithFlags(e, 0); }

hipError_t hipEventRecord(hipEvent_t e, hipStream_t s) {
    if (!e) {
        violation("record of a null event");
        return hipErrorInvalidValue;
    }
    if (s && s->cap) {
        if (s->cap->status != Capture::ACTIVE) {
            violation("record of event %d into capture %d, which is not active", e->id, s->cap->id);
            return hipErrorStreamCaptureInvalidated;
        }
        e->cap = s->cap;
        e->deps = s->deps;
    } else {
        e->cap = nullptr;
        e->deps.clear();
    }
    e->recorded = true;
    return hipSuccess;
}

hipError_t hipStreamWaitEvent(hipStream_t s, hipEvent_t e, unsigned) {
    if (!e) {
        violation("wait on a null event");
        return hipErrorInvalidValue;
    }
    if (!s) {
        if (e->cap)
            violation("the null stream waits on event %d of capture %d", e->id, e->cap->id);
        return hipSuccess;
    }
    if (e->cap) {
        Capture *c = e->cap;
        if (c->status != Capture::ACTIVE) {
            violation("stream %d waits on event %d last recorded in capture %d, which has %s%s",
                      s->id, e->id, c->id, c->status == Capture::ENDED ? "ended" : "been invalidated",
                      c->graph_destroyed ? " and whose graph was destroyed" : "");
            return hipErrorStreamCaptureIsolation;
        }
        if (!s->cap) {  // the stream joins the capture
            s->cap = c;
            s->deps = e->deps;
            c->joined.insert(s);
        } else if (s->cap == c) {
            for (Node *d : e->deps)
                s->deps.push_back(d);
        } else {
            violation("stream %d of capture %d waits on event %d of capture %d (merge)", s->id,
                      s->cap->id, e->id, c->id);
            return hipErrorStreamCaptureMerge;
        }
        return hipSuccess;
    }
    if (s->cap && e->recorded) {
        violation("stream %d of capture %d waits on event %d recorded outside the capture", s->id,
                  s->cap->id, e->id);
        return hipErrorStreamCaptureIsolation;
    }
    return hipSuccess;
}

hipError_t hipEventSynchronize(hipEvent_t e) {
    if (e->cap && e->cap->status == Capture::ACTIVE) {
        violation("synchronize on event %d of active capture %d", e->id, e->cap->id);
        return hipErrorCapturedEvent;
    }
    return hipSuccess;
}

hipError_t hipEventElapsedTime(float *ms, hipEvent_t a, hipEvent_t b) {
    if (a->cap || b->cap)
        violation("elapsed time of events recorded in a capture (%d, %d)", a->id, b->id);
    *ms = 0.f;
    return hipSuccess;
}

hipError_t hipStreamBeginCapture(hipStream_t s, hipStreamCaptureMode) {
    if (!s) {
        violation("capture begun on the null stream");
        return hipErrorStreamCaptureUnsupported;
    }
    if (s->cap) {
        violation("capture begun on stream %d, already in capture %d", s->id, s->cap->id);
        return hipErrorIllegalState;
    }
    auto c = std::make_unique<Capture>();
    c->id = g_next_id++;
    c->origin = s;
    c->joined.insert(s);
    s->cap = c.get();
    s->deps.clear();
    g_captures.push_back(std::move(c));
    return hipSuccess;
}

hipError_t hipStreamEndCapture(hipStream_t s, hipGraph_t *g) {
    *g = nullptr;
    if (!s || !s->cap) {
        violation("capture ended on stream %d, which is not capturing", s ? s->id : 0);
        return hipErrorStreamCaptureUnmatched;
    }
    Capture *c = s->cap;
    if (c->origin != s) {
        violation("capture %d ended on stream %d, not its origin %d", c->id, s->id, c->origin->id);
        return hipErrorStreamCaptureUnmatched;
    }
    std::set<Node *> anc;
    ancestors(s->deps, &anc);
    bool joined = true;
    for (ihipStream_t *j : c->joined) {
        if (j == s)
            continue;
        for (Node *n : j->deps)
            if (!anc.count(n)) {
                violation("capture %d ended while stream %d has work not joined back into the origin",
                          c->id, j->id);
                joined = false;
                break;
            }
    }
    for (ihipStream_t *j : c->joined) {
        j->cap = nullptr;
        j->deps.clear();
    }
    if (!joined || c->status != Capture::ACTIVE) {
        c->status = Capture::INVALID;
        return joined ? hipErrorStreamCaptureInvalidated : hipErrorStreamCaptureUnjoined;
    }
    c->status = Capture::ENDED;
    auto gr = std::make_unique<ihipGraph>();
    gr->cap = c;
    *g = gr.get();
    g_graphs.push_back(std::move(gr));
    return hipSuccess;
}

hipError_t hipGraphInstantiate(hipGraphExec_t *x, hipGraph_t g, hipGraphNode_t *, char *, size_t) {
    if (!g || g->destroyed) {
        violation("instantiation of a null or destroyed graph");
        return hipErrorInvalidValue;
    }
    auto p = std::make_unique<hipGraphExec>();
    p->graph = g;
    p->nodes = (long)g->cap->nodes.size();
    *x = p.get();
    g_execs.push_back(std::move(p));
    return hipSuccess;
}

hipError_t hipGraphLaunch(hipGraphExec_t x, hipStream_t s) {
    if (!x) {
        violation("launch of a null graph");
        return hipErrorInvalidValue;
    }
    return hipsim_enqueue(s, "graph");
}

hipError_t hipGraphDestroy(hipGraph_t g) {
    if (!g || g->destroyed) {
        violation("destroy of a null or destroyed graph");
        return hipErrorInvalidValue;
    }
    g->destroyed = true;
    g->cap->graph_destroyed = true;
    return hipSuccess;
}

hipError_t hipGraphExecDestroy(hipGraphExec_t) { return hipSuccess; }

hipError_t hipGetLastError() { return hipSuccess; }

const char *hipGetErrorString(hipError_t e) {
    switch (e) {
    case hipSuccess: return "hipSuccess";
    case hipErrorStreamCaptureIsolation: return "hipErrorStreamCaptureIsolation";
    case hipErrorStreamCaptureUnjoined: return "hipErrorStreamCaptureUnjoined";
    case hipErrorStreamCaptureMerge: return "hipErrorStreamCaptureMerge";
    case hipErrorStreamCaptureInvalidated: return "hipErrorStreamCaptureInvalidated";
    default: return "hip error";
    }
}
