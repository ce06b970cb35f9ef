// noalloc.hip -- the conv1d backward for callers that cannot allocate device memory:
// its per-row parameter-gradient partials live in a fixed file-scope device array
// instead of a caller workspace.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "launch.hpp"
#include "packmamba.h"

namespace {

constexpr size_t kScratchFloats = PACKMAMBA_NOALLOC_SCRATCH_BYTES / sizeof(float);

// One copy per GPU, held until the process ends.  In host code this name is a
// host-side stand-in, not a device address: the address comes from
// hipGetSymbolAddress, per device.
static __device__ __align__(256) float scratch[kScratchFloats];

constexpr int kMaxDevices = 256;
std::mutex g_mutex;
void* g_scratch[kMaxDevices];   // device address of `scratch` on each device, once looked up

// The current device's address of `scratch`, looked up on the device's first call
// (with that device current) and kept.
int scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return PACKMAMBA_ERR_LAUNCH;
    if (dev >= kMaxDevices) return PACKMAMBA_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_mutex);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return PACKMAMBA_ERR_LAUNCH;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return PACKMAMBA_OK;
}

}  // namespace

extern "C" int packmamba_causal_conv1d_bwd_noalloc(
    const void* x, const float* weight, const float* bias, const int32_t* position_indices,
    const void* initial_x, const void* dout, const void* dfinal_x, void* dx, float* dweight,
    float* dbias, void* dinitial_x, int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
    int32_t dtype, int32_t silu, void* stream) {
    // argument errors and the scratch limit first, with nothing enqueued and the scratch
    // not touched
    if (int e = pm::conv1d_bwd_noalloc_status(x, weight, bias, position_indices, initial_x, dout, dfinal_x, dx,
                                              dweight, dbias, dinitial_x, batch, dim, seqlen, width, dtype))
        return e;
    void* ws = nullptr;
    if (int e = scratch_address(&ws)) return e;
    return packmamba_causal_conv1d_bwd(x, weight, bias, position_indices, initial_x, dout, dfinal_x, dx, dweight,
                                       dbias, dinitial_x, ws, PACKMAMBA_NOALLOC_SCRATCH_BYTES, batch, dim, seqlen,
                                       width, dtype, silu, stream);
}
