// Weight-gradient kernels with fp32 storage, the storage-type dispatch of
// launch_wgrad and the routing-tile check.
#include "wgrad.h"

namespace lstmss {

hipError_t launch_wgrad_bf16(WgradArgs a, bool sparse, hipStream_t s);  // wgrad_bf16.hip

bool wgrad_supported(int P, int R, int S) {
    int greg, tt, at;
    wgrad_tiles(P, R, S, &greg, &tt, &at);
    return tt <= 2 && at <= WG_ATMAX && (R - S) <= 64;
}

hipError_t launch_wgrad(WgradArgs a, bool sparse, bool bf16, hipStream_t s) {
    return bf16 ? launch_wgrad_bf16(a, sparse, s) : launch_wgrad_t<float>(a, sparse, s);
}

} // namespace lstmss
