// Weight-gradient kernels with bf16 storage (fp32 accumulation).
#include "wgrad.h"

namespace lstmss {

hipError_t launch_wgrad_bf16(WgradArgs a, bool sparse, hipStream_t s) {
    return launch_wgrad_t<bf16_t>(a, sparse, s);
}

} // namespace lstmss
