// check_pos.hip -- device check of the position-index contract (§3.1): every row
// starts a sequence (or, for rows that continue a sequence cut at the end of
// another row, starts at any index >= 0), and each later index is 0 or its
// predecessor plus one.
#include "common.hpp"
#include "launch.hpp"

namespace pm {
namespace {

__global__ void check_pos_kernel(const int32_t* __restrict__ pos, int64_t batch, int64_t L,
                                 int32_t continued, int32_t* __restrict__ flag) {
    const int64_t n = batch * L;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t l = i % L;
        const int32_t v = pos[i];
        const bool ok = (l == 0) ? (continued ? v >= 0 : v == 0) : (v == 0 || v == pos[i - 1] + 1);
        if (!ok) *flag = 1;     // every writer stores the same value
    }
}

}  // namespace

hipError_t launch_check_pos(const int32_t* pos, int64_t batch, int64_t seqlen, int32_t continued,
                            int32_t* flag, hipStream_t s) {
    const int64_t n = batch * seqlen;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(check_pos_kernel, dim3((unsigned)blocks), dim3(256), 0, s, pos, batch, seqlen,
                       continued, flag);
    return hipGetLastError();
}

}  // namespace pm
