// rmsnorm.hip -- RMSNorm over the feature axis of (batch, dim, seqlen) activations,
// forward and backward, for the packed Mamba block.  RMSNorm is token-wise, so
// packing leaves it unchanged (§3.2); it is here so that every step of the block
// runs in this library's kernels or in plain GEMMs.
//
// A block of 1024 threads owns a tile of 64 consecutive tokens of one batch row.
// Thread (slice s, group g) holds tokens 8g .. 8g+7 of the tile (one 16-byte bf16
// vector, two fp32 ones) of the features s, s+128, s+256, ...; the 8 groups of a
// slice are consecutive lanes, so each load of a wave reads 8 feature rows of 128
// contiguous bytes.  Many slices keep the loop over the features short, which
// matters for short rows (few tiles).  Per-token sums over the features go through LDS in a fixed
// order.  The second sweep over the tile re-reads its inputs; a tile is
// 64 x dim elements, which the caches hold between the sweeps.
#include "common.hpp"
#include "launch.hpp"

namespace pm {
namespace {

constexpr int kThreads = 1024;
constexpr int kGroups = 8;                   // token groups per tile
constexpr int kTok = 8;                      // tokens per group
constexpr int kTile = kGroups * kTok;        // tokens per tile
constexpr int kSlices = kThreads / kGroups;  // feature slices
static_assert(kTile == kRmsTile, "tile size shared with the workspace sizing");

struct __attribute__((aligned(16))) RmsSmem {
    float red[kSlices][kTile];   // per-slice values of each token
    float tot[kTile];            // their sums
};

// Sum over the slices of each token's per-slice value, in slice order; every
// thread gets its 8 tokens' totals.
__device__ __forceinline__ void slice_sum(float (&v)[kTok], RmsSmem& sm, int sl, int grp) {
    *reinterpret_cast<f32x4*>(&sm.red[sl][grp * kTok]) = f32x4{v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4*>(&sm.red[sl][grp * kTok + 4]) = f32x4{v[4], v[5], v[6], v[7]};
    __syncthreads();
    if (threadIdx.x < kTile) {
        float a = 0.0f;
        for (int q = 0; q < kSlices; ++q) a += sm.red[q][threadIdx.x];
        sm.tot[threadIdx.x] = a;
    }
    __syncthreads();
    const f32x4 a = *reinterpret_cast<const f32x4*>(&sm.tot[grp * kTok]);
    const f32x4 c = *reinterpret_cast<const f32x4*>(&sm.tot[grp * kTok + 4]);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = c.x; v[5] = c.y; v[6] = c.z; v[7] = c.w;
}

template <typename T, typename TO>
__global__ __launch_bounds__(kThreads) void rmsnorm_fwd_kernel(const T* __restrict__ x,
                                                               const float* __restrict__ w, float eps,
                                                               TO* __restrict__ out, float* __restrict__ rstd,
                                                               int64_t dim, int64_t L, int vec) {
    __shared__ RmsSmem sm;
    const int tid = threadIdx.x, grp = tid & (kGroups - 1), sl = tid / kGroups;
    const int64_t b = blockIdx.y;
    const int64_t l0 = (int64_t)blockIdx.x * kTile + grp * kTok;
    const T* xb = x + b * dim * L;
    TO* ob = out + b * dim * L;
    float s[kTok] = {};
    for (int64_t f = sl; f < dim; f += kSlices) {
        float v[kTok];
        load_run<T, kTok>(xb + f * L, l0, L, vec, v);
#pragma unroll
        for (int k = 0; k < kTok; ++k) s[k] = fmaf(v[k], v[k], s[k]);
    }
    slice_sum(s, sm, sl, grp);
    float r[kTok];
#pragma unroll
    for (int k = 0; k < kTok; ++k) r[k] = 1.0f / sqrtf(s[k] / (float)dim + eps);
    if (sl == 0) {
#pragma unroll
        for (int k = 0; k < kTok; ++k)
            if (l0 + k < L) rstd[b * L + l0 + k] = r[k];
    }
    for (int64_t f = sl; f < dim; f += kSlices) {
        float v[kTok];
        load_run<T, kTok>(xb + f * L, l0, L, vec, v);
        const float wf = w[f];
#pragma unroll
        for (int k = 0; k < kTok; ++k) v[k] = v[k] * r[k] * wf;
        store_run<TO, kTok>(ob + f * L, l0, L, vec, v);
    }
}

// dx = r (dh w - x r^2 s / dim) (+ dres), s = sum_f dh w x at each token;
// partial[b, tile, f] = sum over the tile's tokens of dh x r.
template <typename T, typename TO>
__global__ __launch_bounds__(kThreads) void rmsnorm_bwd_kernel(
    const T* __restrict__ x, const float* __restrict__ w, const float* __restrict__ rstd,
    const T* __restrict__ dh, const T* __restrict__ dres, TO* __restrict__ dx,
    float* __restrict__ partial, int64_t dim, int64_t L, int vec) {
    __shared__ RmsSmem sm;
    const int tid = threadIdx.x, grp = tid & (kGroups - 1), sl = tid / kGroups;
    const int64_t b = blockIdx.y;
    const int64_t tile = blockIdx.x;
    const int64_t l0 = tile * kTile + grp * kTok;
    const int64_t off = b * dim * L;
    float s[kTok] = {};
    for (int64_t f = sl; f < dim; f += kSlices) {
        float xv[kTok], gv[kTok];
        load_run<T, kTok>(x + off + f * L, l0, L, vec, xv);
        load_run<T, kTok>(dh + off + f * L, l0, L, vec, gv);
        const float wf = w[f];
#pragma unroll
        for (int k = 0; k < kTok; ++k) s[k] = fmaf(gv[k] * wf, xv[k], s[k]);
    }
    slice_sum(s, sm, sl, grp);
    float r[kTok], c[kTok];
#pragma unroll
    for (int k = 0; k < kTok; ++k) {
        r[k] = (l0 + k < L) ? rstd[b * L + l0 + k] : 0.0f;
        c[k] = r[k] * r[k] * s[k] / (float)dim;
    }
    float* pb = partial + (b * gridDim.x + tile) * dim;
    for (int64_t f = sl; f < dim; f += kSlices) {
        float xv[kTok], gv[kTok], o[kTok];
        load_run<T, kTok>(x + off + f * L, l0, L, vec, xv);
        load_run<T, kTok>(dh + off + f * L, l0, L, vec, gv);
        if (dres) load_run<T, kTok>(dres + off + f * L, l0, L, vec, o);
        const float wf = w[f];
        float pw = 0.0f;
#pragma unroll
        for (int k = 0; k < kTok; ++k) {
            const float v = r[k] * (gv[k] * wf - xv[k] * c[k]);
            o[k] = dres ? o[k] + v : v;
            pw = fmaf(gv[k] * xv[k], r[k], pw);      // 0 past the row end: loads read 0
        }
        store_run<TO, kTok>(dx + off + f * L, l0, L, vec, o);
        // over the 8 groups of the slice (consecutive lanes), in a fixed order
        pw += __shfl_xor(pw, 1, kGroups);
        pw += __shfl_xor(pw, 2, kGroups);
        pw += __shfl_xor(pw, 4, kGroups);
        if (grp == 0) pb[f] = pw;
    }
}

// dw[f] = sum over the (batch, tile) rows of partial[., f], in a fixed order and in two
// passes: a single pass with one thread per feature chained 512 loads per thread at the
// Mamba-1.4B block shape (156 us).  Pass one: block (feature chunk of 64, slab s) sums
// the rows of its slab, each of 4 waves taking every 4th row, and adds the 4 wave sums
// in order; pass two adds the slabs in order.
constexpr int kFinFeat = 64;
__global__ __launch_bounds__(256) void rmsnorm_bwd_finalize_slabs(const float* __restrict__ partial,
                                                                 float* __restrict__ slabs, int64_t rows,
                                                                 int64_t dim) {
    __shared__ float part[4][kFinFeat];
    const int fo = threadIdx.x & (kFinFeat - 1), rg = threadIdx.x / kFinFeat;
    const int64_t f = (int64_t)blockIdx.x * kFinFeat + fo;
    const int64_t per = (rows + kRmsSlabs - 1) / kRmsSlabs;
    const int64_t i0 = (int64_t)blockIdx.y * per, i1 = min(rows, i0 + per);
    float a = 0.0f;
    if (f < dim)
        for (int64_t i = i0 + rg; i < i1; i += 4) a += partial[i * dim + f];
    part[rg][fo] = a;
    __syncthreads();
    if (rg == 0 && f < dim) slabs[blockIdx.y * dim + f] = ((part[0][fo] + part[1][fo]) + part[2][fo]) + part[3][fo];
}

__global__ void rmsnorm_bwd_finalize(const float* __restrict__ slabs, float* __restrict__ dw, int64_t dim) {
    const int64_t f = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (f >= dim) return;
    float a = 0.0f;
#pragma unroll
    for (int q = 0; q < kRmsSlabs; ++q) a += slabs[q * dim + f];
    dw[f] = a;
}

template <typename T, typename TO>
hipError_t fwd_t(const RmsArgs& a, hipStream_t s) {
    const int vec = (a.seqlen % Storage<T>::kPerVec) == 0 && (a.seqlen % Storage<TO>::kPerVec) == 0;
    const dim3 grid((unsigned)((a.seqlen + kTile - 1) / kTile), (unsigned)a.batch);
    hipLaunchKernelGGL((rmsnorm_fwd_kernel<T, TO>), grid, dim3(kThreads), 0, s, static_cast<const T*>(a.x),
                       a.w, a.eps, static_cast<TO*>(a.out), a.rstd_out, a.dim, a.seqlen, vec);
    return hipGetLastError();
}

template <typename T, typename TO>
hipError_t bwd_t(const RmsArgs& a, hipStream_t s) {
    const int vec = (a.seqlen % Storage<T>::kPerVec) == 0 && (a.seqlen % Storage<TO>::kPerVec) == 0;
    const int64_t tiles = (a.seqlen + kTile - 1) / kTile;
    const dim3 grid((unsigned)tiles, (unsigned)a.batch);
    hipLaunchKernelGGL((rmsnorm_bwd_kernel<T, TO>), grid, dim3(kThreads), 0, s, static_cast<const T*>(a.x),
                       a.w, a.rstd, static_cast<const T*>(a.dout), static_cast<const T*>(a.dres),
                       static_cast<TO*>(a.out), a.partial, a.dim, a.seqlen, vec);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    float* slabs = a.partial + a.batch * tiles * a.dim;
    hipLaunchKernelGGL(rmsnorm_bwd_finalize_slabs, dim3((unsigned)((a.dim + kFinFeat - 1) / kFinFeat), kRmsSlabs),
                       dim3(256), 0, s, a.partial, slabs, a.batch * tiles, a.dim);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(rmsnorm_bwd_finalize, dim3((unsigned)((a.dim + 255) / 256)), dim3(256), 0, s,
                       slabs, a.dw, a.dim);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_rmsnorm_fwd(const RmsArgs& a, hipStream_t s) {
    switch (a.dtype) {
        case 1: return fwd_t<bf16_t, bf16_t>(a, s);
        case 2: return fwd_t<bf16_t, float>(a, s);
        default: return fwd_t<float, float>(a, s);
    }
}

hipError_t launch_rmsnorm_bwd(const RmsArgs& a, hipStream_t s) {
    switch (a.dtype) {
        case 1: return bwd_t<bf16_t, bf16_t>(a, s);
        case 2: return bwd_t<bf16_t, float>(a, s);
        default: return bwd_t<float, float>(a, s);
    }
}

}  // namespace pm
