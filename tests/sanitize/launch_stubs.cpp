// Stand-ins for the kernel launchers, for the host-only sanitizer build of the C ABI
// (api.cpp, pack.cpp) that runs on a machine without a GPU: every launch reports
// failure, so an argument check that lets a bad call through shows up as
// PACKMAMBA_ERR_LAUNCH instead of the expected error.  Test infrastructure only.
#include "launch.hpp"
#include "packmamba.h"

namespace pm {
hipError_t launch_conv1d_fwd(const ConvArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_conv1d_bwd(const ConvArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_rmsnorm_fwd(const RmsArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_rmsnorm_bwd(const RmsArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_scan_fwd(const ScanArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_scan_bwd(const ScanArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_check_pos(const int32_t*, int64_t, int64_t, int32_t, int32_t*, hipStream_t) {
    return hipErrorInvalidValue;
}
}  // namespace pm

// The no-allocation entry point without its device-symbol part: the same host checks,
// then a failed launch.
extern "C" int packmamba_causal_conv1d_bwd_noalloc(
    const void* x, const float* weight, const float* bias, const int32_t* position_indices,
    const void* initial_x, const void* dout, const void* dfinal_x, void* dx, float* dweight,
    float* dbias, void* dinitial_x, int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
    int32_t dtype, int32_t, void*) {
    if (int e = pm::conv1d_bwd_noalloc_status(x, weight, bias, position_indices, initial_x, dout, dfinal_x, dx,
                                              dweight, dbias, dinitial_x, batch, dim, seqlen, width, dtype))
        return e;
    return PACKMAMBA_ERR_LAUNCH;
}
