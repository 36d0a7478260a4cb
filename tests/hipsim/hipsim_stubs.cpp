// Stand-ins for the library's kernel launchers when its host driver is built
// against the stream-capture model: every launch becomes one work item on its
// stream.  The host-side shape rules that decide which launches a call makes
// (split gate path, data-gradient tiles, weight-gradient support) follow the
// library's own rules.
#include "../../paper_1806_00512_amd/csrc/kernels.h"

#include <algorithm>

extern "C" int hipsim_enqueue(hipStream_t s, const char *what);

namespace lstmss {

static hipError_t item(hipStream_t s, const char *what) { return hipsim_enqueue(s, what); }

hipError_t launch_cell(const CellArgs &, int, bool, hipStream_t s) { return item(s, "cell"); }
hipError_t launch_cell_fine(const CellArgs &, int, bool, hipStream_t s) { return item(s, "cell_fine"); }
size_t cell_lds_bytes(const CellArgs &, int) { return 1024; }
bool cell_split_ok(const CellArgs &a, int mode) {
    if ((long)a.H * a.B < 65536)
        return false;
    return mode == CELL_DENSE ||
           ((long)a.regions_per_wg * a.R <= 64 && (long)a.regions_per_wg * a.R * a.P <= 256);
}
hipError_t launch_bias_grad(float *, const float *, int, long, int, int, const int32_t *, int, int,
                            int, int, bool, hipStream_t s) {
    return item(s, "bias_grad");
}
hipError_t launch_gemm1(Gemm1Args, bool, hipStream_t s) { return item(s, "gemm1"); }
bool gemm1_select_ok(Gemm1Args a, bool bf16) {
    const int R = a.sel_R, S = a.sel_S;
    return a.sel_sq && a.steps == 1 && R >= 1 && R <= 64 && S >= 1 && S < R &&
           a.Kp % (bf16 ? 64 : 32) == 0 && a.k_chunk <= GEMM1_KC_MAX &&
           a.k_chunk % ((long)a.P * (R - S)) == 0;
}
hipError_t launch_gemm2(const Gemm2Args &, bool, hipStream_t s) { return item(s, "gemm2"); }
hipError_t launch_gemm_fwd(Gemm1Args, bool, hipStream_t s) { return item(s, "gemm_fwd"); }
hipError_t launch_fwd_act(const FwdActArgs &, bool, hipStream_t s) { return item(s, "fwd_act"); }
hipError_t launch_sgd(void *, const float *, long, float *, const float *, long, float, bool,
                      hipStream_t s) {
    return item(s, "sgd");
}
hipError_t launch_mse(const void *, const float *, float *, long, float, double *, int, bool,
                      hipStream_t s) {
    return item(s, "mse");
}
hipError_t launch_reverse(const void *, void *, int, long, hipStream_t s) { return item(s, "reverse"); }
hipError_t launch_bidir_join(const void *, const void *, void *, int, long, bool, hipStream_t s) {
    return item(s, "bidir_join");
}
hipError_t launch_bidir_split(const float *, float *, float *, int, long, hipStream_t s) {
    return item(s, "bidir_split");
}
hipError_t launch_sum_rev(const float *, const float *, float *, int, long, hipStream_t s) {
    return item(s, "sum_rev");
}
hipError_t launch_wgrad(WgradArgs, bool, bool, hipStream_t s) { return item(s, "wgrad"); }
bool wgrad_supported(int P, int R, int S) {
    const int kr = (R - S) * P, rp = R * P;
    const int greg = kr <= 32 ? std::max(1, 32 / kr) : 1;
    return (greg * kr + 31) / 32 <= 2 && (greg * rp + 31) / 32 <= 4 && R - S <= 64;
}
hipError_t launch_fwd_step(const FwdArgs &, bool, hipStream_t s) { return item(s, "fwd_step"); }
hipError_t launch_fill(float *, long, float, hipStream_t s) { return item(s, "fill"); }
hipError_t launch_copy_in(float *, const float *, long, hipStream_t s) { return item(s, "copy_in"); }
hipError_t launch_reduce_parts(float *, const float *, int, long, long, hipStream_t s) {
    return item(s, "reduce_parts");
}
hipError_t launch_h0_store(void *, const float *, long, bool, hipStream_t s) { return item(s, "h0_store"); }
void gemm1_tile(bool bf16, int N, long rows, long zdim, int *tm, int *tn) {
    if (N <= 32) {
        *tm = 128;
        *tn = 32;
    } else if (N <= 64) {
        *tm = bf16 ? 128 : 64;
        *tn = 64;
    } else if (bf16 || ((rows + 127) / 128) * ((N + 127) / 128) * zdim >= 256) {
        *tm = 128;
        *tn = 128;
    } else {
        *tm = 64;
        *tn = 64;
    }
}
int gemm1_wgs_per_cu(int tm, int tn) {
    const long lds = 2L * (tm + tn) * 144 + 4L * GEMM1_KC_MAX;
    return (int)std::max(1L, (160L * 1024) / lds);
}

} // namespace lstmss
