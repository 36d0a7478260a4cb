// The entry point that allocates nothing: the standalone selection with its
// scratch (the per-row, per-64-column-chunk fp64 sums of squares of the
// two-kernel gate path) in a static device array instead of a caller
// workspace.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <map>
#include <mutex>

#include "kernels.h"

namespace {

// Every GPU the library runs on holds its own copy of this array until the
// process ends.  In host code its name stands for a host-side shadow, not a
// device address: the device address of the current GPU's copy comes from
// hipGetSymbolAddress (scratch_on_device) and is the only form passed on.
constexpr size_t kScratchBytes = LSTMSS_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
std::map<int, void *> g_scratch_ptr;  // device ordinal -> its copy of `scratch`

// Device address of the current device's copy, looked up once per device
// (with that device current) and kept.
hipError_t scratch_on_device(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    auto it = g_scratch_ptr.find(dev);
    if (it != g_scratch_ptr.end()) {
        *out = it->second;
        return hipSuccess;
    }
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess)
        return e;
    if (!p)
        return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
    *out = p;
    return hipSuccess;
}

} // namespace

extern "C" int32_t lstmss_select_compact_noalloc(const lstmss_dims *d, float sparsity,
                                                 const lstmss_structure *s, const void *dG,
                                                 void *dG_c, int32_t *idx, double *scores,
                                                 void *stream) {
    // size first (before any pointer is looked at): nothing is launched for
    // a shape whose scratch would not fit
    const int64_t need = lstmss::select_scratch_bytes(d, sparsity, s);
    if (need < 0)
        return (int32_t)need;
    if ((size_t)need > kScratchBytes) {
        char msg[160];
        snprintf(msg, sizeof(msg),
                 "the selection needs %lld bytes of scratch; the static buffer holds %zu "
                 "(4H * ceil(B/64) * 8 bytes must fit)",
                 (long long)need, kScratchBytes);
        return lstmss::set_error(LSTMSS_ERR_UNSUPPORTED, msg);
    }
    void *ws = nullptr;
    if (need > 0) {
        const hipError_t e = scratch_on_device(&ws);
        if (e != hipSuccess) {
            char msg[160];
            snprintf(msg, sizeof(msg), "hipGetSymbolAddress(scratch) failed: %s",
                     hipGetErrorString(e));
            return lstmss::set_error(LSTMSS_ERR_HIP, msg);
        }
    }
    return lstmss::select_compact_impl(d, sparsity, s, dG, dG_c, idx, scores, ws, (size_t)need,
                                       stream, false);
}
