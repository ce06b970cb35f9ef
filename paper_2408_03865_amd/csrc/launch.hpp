// launch.hpp -- host-side launchers of the gfx950 kernels, called by the C ABI
// after argument validation.  Each returns hipSuccess or the launch error.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pm {

struct ConvArgs {
    const void* x;
    const float* w;
    const float* bias;
    const int32_t* pos;
    const void* dout;   // bwd only
    void* out;          // fwd: out; bwd: dx
    float* dw;          // bwd only
    float* dbias;       // bwd only
    float* partial;     // bwd only: (batch, segments, dim, width+1)
    // state passing across rows, each (batch, dim, width-1) or null
    const void* xinit;  // inputs before the row (x's dtype)
    void* xfinal;       // fwd: the row's last width-1 inputs (x's dtype)
    const void* dxfinal;// bwd: gradient of xfinal (dout's dtype)
    void* dxinit;       // bwd: gradient of xinit (dx's dtype)
    int64_t batch, dim, seqlen;
    int32_t width, dtype, silu;
};

hipError_t launch_conv1d_fwd(const ConvArgs& a, hipStream_t s);
// Argument checks of packmamba_causal_conv1d_bwd other than its workspace (a status code).
int conv1d_bwd_args_status(const void* x, const float* weight, const float* bias, const int32_t* position_indices,
                           const void* initial_x, const void* dout, const void* dfinal_x, const void* dx,
                           const float* dweight, const float* dbias, const void* dinitial_x, int64_t batch,
                           int64_t dim, int64_t seqlen, int32_t width, int32_t dtype);
// The same plus the no-allocation variant's limit: PACKMAMBA_ERR_SCRATCH when the shape's
// workspace exceeds its fixed scratch.
int conv1d_bwd_noalloc_status(const void* x, const float* weight, const float* bias,
                              const int32_t* position_indices, const void* initial_x, const void* dout,
                              const void* dfinal_x, const void* dx, const float* dweight, const float* dbias,
                              const void* dinitial_x, int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
                              int32_t dtype);
hipError_t launch_conv1d_bwd(const ConvArgs& a, hipStream_t s);

// RMSNorm over the feature axis of (batch, dim, seqlen) activations.
constexpr int64_t kRmsTile = 64;     // tokens per block; one dweight partial per (batch, tile)
constexpr int kRmsSlabs = 16;        // row slabs of the dweight reduction's first pass
struct RmsArgs {
    const void* x;
    const float* w;
    const float* rstd;  // bwd: saved by the forward, (batch, seqlen)
    const void* dout;   // bwd only
    const void* dres;   // bwd only: gradient added to dx, or null
    void* out;          // fwd: out; bwd: dx
    float* rstd_out;    // fwd: (batch, seqlen)
    float* dw;          // bwd only
    float* partial;     // bwd only: (batch, tiles, dim), then (kRmsSlabs, dim) slab sums
    float eps;
    int64_t batch, dim, seqlen;
    int32_t dtype;
};
hipError_t launch_rmsnorm_fwd(const RmsArgs& a, hipStream_t s);
hipError_t launch_rmsnorm_bwd(const RmsArgs& a, hipStream_t s);

// The conv backward runs one wave per (row, segment); a row is cut into segments of
// whole 512-token steps when batch x dim alone gives fewer than kConvBwdWaves waves.
constexpr int64_t kConvBwdSpan = 512;
constexpr int64_t kConvBwdWaves = 4096;
inline int64_t conv_bwd_segments(int64_t batch, int64_t dim, int64_t seqlen) {
    const int64_t steps = (seqlen + kConvBwdSpan - 1) / kConvBwdSpan;
    const int64_t rows = batch * dim;
    int64_t nseg = (kConvBwdWaves + rows - 1) / rows;
    if (nseg > steps) nseg = steps;
    if (nseg < 1) nseg = 1;
    const int64_t per = (steps + nseg - 1) / nseg;       // steps per segment
    return (steps + per - 1) / per;                     // no empty segment
}

struct ScanArgs {
    const void* u;
    const void* delta;
    const float* A;
    const void* B;
    const void* C;
    const float* D;
    const void* z;
    const float* delta_bias;
    const int32_t* pos;
    int32_t softplus;
    // state passing across rows, each (batch, dim, dstate) fp32 or null
    const float* h0;        // state before the row
    float* hfinal;          // fwd: state after the row
    const float* dhfinal;   // bwd: gradient of hfinal
    float* dh0;             // bwd: gradient of h0
    // forward
    void* out;
    float* states;          // (batch, dim, nchunk, dstate); written by fwd, read by bwd
    float* dzf;             // (batch, dim, seqlen): (y + D u) d(z sigmoid(z))/dz, the factor of
                            // dout in dz; written by fwd beside the states when z is given,
                            // read by bwd (required there when z is given)
    // backward
    const void* dout;
    void* du;
    void* ddelta;
    void* dz;
    float* dA;
    float* dB;
    float* dC;
    float* dD;
    float* ddelta_bias;
    float* part_bc;         // (batch, groups, 2, dstate, seqlen)
    float* part_chan;       // (batch, nseg, dim, dstate + 2)
    // segment split (both directions): per-segment maps and the chained carries
    float* ws_agg;          // (batch, dim, nseg, dstate, 2)
    float* ws_carry;        // (batch, dim, nseg, dstate)
    int64_t batch, dim, seqlen;
    int32_t dstate, dtype;
};

// The factor of dout in dz, saved by the scan forward for the backward (fp32): each
// (batch, channel) row is padded to whole chunks of kDzfChunk = 256 tokens
// (dzf_row_len), and a chunk is stored as [i][lane][q] for its token 16 lane + 4 i + q.
// The forward's lane holds 16 consecutive tokens, and its i-th 16-byte store lands
// beside the other lanes' i-th stores, so every store instruction writes whole
// 128-byte lines of a row; the backward's 8-token run (lane j of a 128-token chunk)
// is two such vectors, also whole lines per wave.
constexpr int64_t kDzfChunk = 256;
__host__ __device__ constexpr int64_t dzf_row_len(int64_t L) {
    return (L + kDzfChunk - 1) / kDzfChunk * kDzfChunk;
}
// float offset, inside a padded row, of vector i (tokens 4 i .. 4 i + 3) of lane j's
// 16 tokens in 256-token chunk c
__host__ __device__ constexpr int64_t dzf_vec(int64_t c, int i, int j) {
    return c * kDzfChunk + (i * 16 + j) * 4;
}

// channels reduced on chip per dB/dC partial in the backward
constexpr int kScanBwdChannels = 16;

// Split of the rows into segments along the sequence, each scanned by its own
// block with the carry across segments resolved by an aggregate pass and a carry
// pass.  Used only when batch x (channel groups of 16) leaves the GPU underfilled:
// 256 CUs hold three scan blocks each.  A direction splits when its blocks fill less
// than half of its target and then aims at the target: one round of blocks (768) for
// the forward, two (1536) for the backward, each direction's fastest (4 rows x 2048
// tokens x 1536 channels, 384 blocks: the forward unsplit takes 102 us against 115 us
// in 4 segments, while the backward gains from its 4).  More segments never need less
// workspace, so the backward's plan also covers the forward's recompute.
struct SegPlan {
    int64_t nseg;      // segments per row (1: no split)
    int64_t seg_len;   // tokens per segment, a multiple of kSegUnit
};
constexpr int64_t kSegUnit = 256;          // forward chunk, a multiple of the backward chunk
constexpr int64_t kSegTargetFwd = 768;
constexpr int64_t kSegTargetBwd = 1536;

inline SegPlan scan_segments(int64_t batch, int64_t dim, int64_t seqlen, int64_t target) {
    const int64_t blocks = batch * ((dim + 15) / 16);
    const int64_t units = (seqlen + kSegUnit - 1) / kSegUnit;
    if (blocks * 2 >= target || units < 2) return {1, units * kSegUnit};
    int64_t nseg = (target + blocks - 1) / blocks;
    if (nseg > units) nseg = units;
    const int64_t per = (units + nseg - 1) / nseg;
    return {(units + per - 1) / per, per * kSegUnit};
}

hipError_t launch_scan_fwd(const ScanArgs& a, hipStream_t s);
hipError_t launch_scan_bwd(const ScanArgs& a, hipStream_t s);
hipError_t launch_check_pos(const int32_t* pos, int64_t batch, int64_t seqlen, int32_t continued,
                            int32_t* flag, hipStream_t s);

}  // namespace pm
