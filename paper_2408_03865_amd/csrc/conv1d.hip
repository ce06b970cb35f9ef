// conv1d.hip -- packed causal depthwise conv1d, forward and backward (Alg. 1, §3.3, §3.5).
//
// HBM-bound streaming kernels.  The tap mask uses only integer compares against
// the token's position index, read with the same coalesced vector loads (§3.5):
// the forward keeps the tap reaching k tokens back iff k <= pos[l]; the
// backward's dx takes the next width-1 tokens' indices ("reverse indices") and
// keeps tap k iff pos[j+k] >= k.
//  - Forward: one 256-thread block per (batch, channel) row; each thread owns 8
//    consecutive tokens per step (one 16-byte vector of bf16, two of fp32) and
//    loops along the row.  The width-1 halo comes from the neighbouring vector,
//    which the neighbouring lane loads in the same instruction, so it is served by
//    the cache and costs no extra HBM traffic.
//  - Backward: one wave per (row, segment), described at its kernel.
#include "common.hpp"
#include "launch.hpp"

namespace pm {
namespace {

constexpr int kTok = 8;        // tokens per thread per step (forward), and the halo vector
constexpr int kTokBwd = 8;     // tokens per thread per step (backward)
constexpr int kThreads = 256;

// N position indices from l0 (N a multiple of 4); beyond L they read 0.  FULL: the
// caller guarantees l0 + N <= L and 16-byte alignment
template <int N = kTok, bool FULL = false>
__device__ __forceinline__ void load_pos(const int32_t* __restrict__ pr, int64_t l0, int64_t L,
                                         bool pvec, int* p) {
    if (FULL || (pvec && l0 + N <= L)) {
#pragma unroll
        for (int i = 0; i < N; i += 4) {
            const u32x4 a = *reinterpret_cast<const u32x4*>(pr + l0 + i);
            p[i] = (int)a.x; p[i + 1] = (int)a.y; p[i + 2] = (int)a.z; p[i + 3] = (int)a.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < N; ++i) p[i] = (l0 + i < L) ? pr[l0 + i] : 0;
    }
}

// Per-row states of a sequence cut at a row end (§5): (batch*dim, W-1) arrays, or
// null.  xinit holds the W-1 inputs before the row (token -1 last), xfinal the
// row's last W-1 inputs; dxfinal and dxinit are their gradients.
template <typename T, typename TO>
struct ConvStates {
    const T* xinit;
    T* xfinal;
    const T* dxfinal;
    TO* dxinit;
};

// The W-1 tokens before the row into xs[kTok-W+1 .. kTok-1] (zeros without xinit).
template <typename T, int W>
__device__ __forceinline__ void load_row_halo(const T* __restrict__ xinit, int64_t row, float* xs) {
#pragma unroll
    for (int i = 0; i < kTok; ++i) xs[i] = 0.0f;
    if (xinit) {
#pragma unroll
        for (int t = 0; t < W - 1; ++t) xs[kTok - (W - 1) + t] = Storage<T>::load1(xinit + row * (W - 1) + t);
    }
}

// pre-activation of the token at index i of `xs`, where xs[kTok + t] holds token
// l0 + t and xs[kTok - 1 - t] holds token l0 - 1 - t
template <int W>
__device__ __forceinline__ float conv_pre(const float* xs, int i, int p, const float* wk, float b0) {
    float acc = fmaf(wk[W - 1], xs[kTok + i], b0);      // tap 0: position indices are >= 0
#pragma unroll
    for (int k = 1; k < W; ++k)
        if (k <= p) acc = fmaf(wk[W - 1 - k], xs[kTok + i - k], acc);
    return acc;
}

template <typename T, typename TO, int W>
__global__ __launch_bounds__(kThreads) void conv1d_fwd_kernel(
    const T* __restrict__ x, const float* __restrict__ w, const float* __restrict__ bias,
    const int32_t* __restrict__ pos, TO* __restrict__ out, ConvStates<T, TO> st, int64_t dim,
    int64_t L, int silu, int vec, int pvec) {
    const int64_t row = blockIdx.x;
    const int64_t b = row / dim, d = row - b * dim;
    const T* xr = x + row * L;
    TO* orow = out + row * L;
    const int32_t* pr = pos + b * L;
    float wk[W];
#pragma unroll
    for (int k = 0; k < W; ++k) wk[k] = w[d * W + k];
    const float b0 = bias ? bias[d] : 0.0f;

    for (int64_t l0 = (int64_t)threadIdx.x * kTok; l0 < L; l0 += (int64_t)kThreads * kTok) {
        float xs[2 * kTok];
        load_run<T, kTok>(xr, l0, L, vec, xs + kTok);
        if (l0 > 0) load_run<T, kTok>(xr, l0 - kTok, L, vec, xs);
        else load_row_halo<T, W>(st.xinit, row, xs);
        int p[kTok];
        load_pos(pr, l0, L, pvec, p);
        float o[kTok];
#pragma unroll
        for (int i = 0; i < kTok; ++i) {
            const float v = conv_pre<W>(xs, i, p[i], wk, b0);
            o[i] = silu ? v * sigmoid_f(v) : v;
        }
        store_run<TO, kTok>(orow, l0, L, vec, o);
    }
    // the row's last W-1 inputs, copied as stored (reaching into xinit for short rows)
    if (st.xfinal && threadIdx.x == 0) {
#pragma unroll
        for (int i = 0; i < W - 1; ++i) {
            const int64_t m = L - (W - 1) + i;
            T v{};
            if (m >= 0) v = xr[m];
            else if (st.xinit) v = st.xinit[row * (W - 1) + (W - 1) + m];
            st.xfinal[row * (W - 1) + i] = v;
        }
    }
}

// Backward: one wave per (row, segment), walking the segment from its end in steps
// of 64*KT tokens (long rows with few channels are cut into segments of whole steps,
// so that the grid has enough waves).
// Each lane owns KT consecutive tokens per step and computes their activation
// gradient g once.  dx of a token needs g of the next W-1 tokens (the reverse-index
// halo): they belong to the next lane, which hands over their masked values with a
// lane shift, and for lane 63 to lane 0 of the previous (later) step, whose values
// are carried.
// DXF: a final-input gradient is given (a separate instantiation, so that the
// common path keeps its register count).
template <typename T, typename TO, int W, int KT, bool DXF>
__global__ __launch_bounds__(64) void conv1d_bwd_kernel(
    const T* __restrict__ x, const float* __restrict__ w, const float* __restrict__ bias,
    const int32_t* __restrict__ pos, const T* __restrict__ dout, TO* __restrict__ dx,
    float* __restrict__ partial, ConvStates<T, TO> st, int64_t dim, int64_t L, int silu, int vec,
    int pvec) {
    static_assert(KT >= W - 1 && KT % 4 == 0, "the halo lies in the next lane's tokens");
    const int64_t row = blockIdx.x;
    const int64_t b = row / dim, d = row - b * dim;
    const int seg = blockIdx.y, nseg = gridDim.y;
    const int lane = (int)threadIdx.x;
    const T* xr = x + row * L;
    const T* gr = dout + row * L;
    TO* dxr = dx + row * L;
    const int32_t* pr = pos + b * L;
    float wk[W];
#pragma unroll
    for (int k = 0; k < W; ++k) wk[k] = w[d * W + k];
    const float b0 = bias ? bias[d] : 0.0f;
    constexpr int64_t kSpan = 64 * KT;
    static_assert(kSpan == kConvBwdSpan, "segments hold whole steps");
    const int64_t nsteps = (L + kSpan - 1) / kSpan;
    const int64_t seg_steps = (nsteps + nseg - 1) / nseg;
    const int64_t s0 = (int64_t)seg * seg_steps;
    const int64_t s1 = min(nsteps, s0 + seg_steps);
    float acc[W + 1];   // dw[0..W-1], dbias
#pragma unroll
    for (int j = 0; j <= W; ++j) acc[j] = 0.0f;
    // masked activation gradients gm[k][t] (k > t, t < W-1) of the first W-1 tokens of
    // lane 0 in the step to the right: 0 past the row end; at the end of a segment that
    // is not the row's last, recomputed here (the same value in every lane)
    float cgm[W][W - 1];
#pragma unroll
    for (int k = 0; k < W; ++k) {
#pragma unroll
        for (int t = 0; t < W - 1; ++t) cgm[k][t] = 0.0f;
    }
    if (s1 * kSpan < L) {
        const int64_t e = s1 * kSpan;               // first token after the segment
#pragma unroll
        for (int t = 0; t < W - 1; ++t) {
            const int64_t l = e + t;
            if (l >= L) break;
            const int p = pr[l];
            float g = Storage<T>::load1(gr + l);
            if (silu) {
                float v = b0;
#pragma unroll
                for (int k = 0; k < W; ++k)
                    if (k <= p) v = fmaf(wk[W - 1 - k], Storage<T>::load1(xr + l - k), v);
                const float sg = sigmoid_f(v);
                g *= sg * (1.0f + v * (1.0f - sg));
            }
#pragma unroll
            for (int k = t + 1; k < W; ++k) cgm[k][t] = k <= p ? g : 0.0f;
        }
    }
    // One step; FULL (wave-uniform) means the step lies inside the row and vector access
    // is allowed, so the loads and stores need no bounds checks.
    auto step = [&](auto full_tag, const int64_t sidx) {
        constexpr bool FULL = decltype(full_tag)::value;
        const int64_t l0 = sidx * kSpan + (int64_t)lane * KT;
        // x of tokens l0-8 .. l0+KT-1 (pre-activations of this lane's tokens)
        float xs[kTok + KT];
        if (l0 > 0) load_run<T, kTok, FULL>(xr, l0 - kTok, L, vec, xs);
        else load_row_halo<T, W>(st.xinit, row, xs);
        load_run<T, KT, FULL>(xr, l0, L, vec, xs + kTok);
        float gs[KT];
        load_run<T, KT, FULL>(gr, l0, L, vec, gs);   // 0 beyond L, so g = 0 there
        int p[KT];
        load_pos<KT, FULL>(pr, l0, L, pvec, p);
        // gm[k][t] = g[t] if tap k of token t is live (k <= pos[t]) else 0, with g the
        // activation gradient.  The same masked values give dx through the reverse
        // indices (tap k of token j is live iff pos[j+k] >= k) and dw.  Tap 0 is always
        // live (position indices are >= 0).
        float gm[W][KT + W - 1];
#pragma unroll
        for (int t = 0; t < KT; ++t) {
            bool live[W];
#pragma unroll
            for (int k = 1; k < W; ++k) live[k] = k <= p[t];
            float gt = gs[t];
            if (silu) {
                float v = fmaf(wk[W - 1], xs[kTok + t], b0);
#pragma unroll
                for (int k = 1; k < W; ++k)
                    if (live[k]) v = fmaf(wk[W - 1 - k], xs[kTok + t - k], v);
                const float sg = sigmoid_f(v);
                gt *= sg * (1.0f + v * (1.0f - sg));
            }
            gm[0][t] = gt;
#pragma unroll
            for (int k = 1; k < W; ++k) gm[k][t] = live[k] ? gt : 0.0f;
        }
        // the next W-1 tokens (only the taps that reach back into this lane): from the
        // next lane, or for lane 63 from the carry; then lane 0's become the carry
#pragma unroll
        for (int t = 0; t < W - 1; ++t) {
#pragma unroll
            for (int k = t + 1; k < W; ++k) {
                const float h = __shfl_down(gm[k][t], 1, 64);
                gm[k][KT + t] = lane == 63 ? cgm[k][t] : h;
                cgm[k][t] = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, gm[k][t])));
            }
        }
        float o[KT];
#pragma unroll
        for (int i = 0; i < KT; ++i) {
            float a = wk[W - 1] * gm[0][i];
#pragma unroll
            for (int k = 1; k < W; ++k) a = fmaf(wk[W - 1 - k], gm[k][i + k], a);
            o[i] = a;
        }
        // the final inputs are copies of the last W-1 inputs: their gradient adds in
        if (DXF && l0 + KT > L - (W - 1)) {
#pragma unroll
            for (int i = 0; i < KT; ++i) {
                const int64_t j = l0 + i - (L - (W - 1));
                if (j >= 0 && l0 + i < L) o[i] += Storage<T>::load1(st.dxfinal + row * (W - 1) + j);
            }
        }
        store_run<TO, KT, FULL>(dxr, l0, L, vec, o);
        // parameter gradients from this lane's own tokens
#pragma unroll
        for (int i = 0; i < KT; ++i) {
#pragma unroll
            for (int k = 0; k < W; ++k) acc[W - 1 - k] = fmaf(gm[k][i], xs[kTok + i - k], acc[W - 1 - k]);
            acc[W] += gm[0][i];
        }
    };
    for (int64_t sidx = s1 - 1; sidx >= s0; --sidx) {
        if (vec && pvec && (sidx + 1) * kSpan <= L) step(std::true_type{}, sidx);
        else step(std::false_type{}, sidx);
    }
    // gradient of the inputs before the row: initial input j (token j-W+1) meets output
    // token t <= j through tap k = t-j+W-1 > t (weight w[j-t]); the carry now holds the
    // masked gradients of tokens 0..W-2
    if (st.dxinit && seg == 0 && lane == 0) {
#pragma unroll
        for (int j = 0; j < W - 1; ++j) {
            float a = 0.0f;
#pragma unroll
            for (int t = 0; t <= j; ++t) a = fmaf(wk[j - t], cgm[t - j + W - 1][t], a);
            // a row shorter than W-1 copies initial input j >= L to final input j - L
            if (st.dxfinal && j >= L) a += Storage<T>::load1(st.dxfinal + row * (W - 1) + (j - L));
            Storage<TO>::store1(st.dxinit + row * (W - 1) + j, a);
        }
    }
#pragma unroll
    for (int j = 0; j <= W; ++j) {
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) acc[j] += __shfl_xor(acc[j], off, 64);
    }
    if (lane == 0) {
        float* pp = partial + ((b * nseg + seg) * dim + d) * (W + 1);
#pragma unroll
        for (int j = 0; j <= W; ++j) pp[j] = acc[j];
    }
}

// dw[d,k] = sum_r partial[r,d,k]; dbias[d] = sum_r partial[r,d,W] over the (batch row,
// segment) pairs r, in a fixed order
__global__ void conv1d_bwd_finalize(const float* __restrict__ partial, float* __restrict__ dw,
                                    float* __restrict__ dbias, int64_t batch, int64_t dim, int W) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= dim * (W + 1)) return;
    const int64_t d = i / (W + 1);
    const int j = (int)(i - d * (W + 1));
    float s = 0.0f;
    for (int64_t b = 0; b < batch; ++b) s += partial[(b * dim + d) * (W + 1) + j];
    if (j < W) dw[d * W + j] = s;
    else if (dbias) dbias[d] = s;
}

template <typename T, typename TO>
hipError_t conv_fwd_t(const ConvArgs& a, hipStream_t s) {
    const int vec = (a.seqlen % Storage<T>::kPerVec) == 0 && (a.seqlen % Storage<TO>::kPerVec) == 0;
    const int pvec = (a.seqlen % 4) == 0;
    dim3 grid((unsigned)(a.batch * a.dim)), block(kThreads);
    const T* x = static_cast<const T*>(a.x);
    TO* o = static_cast<TO*>(a.out);
    const ConvStates<T, TO> st{static_cast<const T*>(a.xinit), static_cast<T*>(a.xfinal), nullptr, nullptr};
    switch (a.width) {
        case 2: hipLaunchKernelGGL((conv1d_fwd_kernel<T, TO, 2>), grid, block, 0, s, x, a.w, a.bias, a.pos, o, st, a.dim, a.seqlen, a.silu, vec, pvec); break;
        case 3: hipLaunchKernelGGL((conv1d_fwd_kernel<T, TO, 3>), grid, block, 0, s, x, a.w, a.bias, a.pos, o, st, a.dim, a.seqlen, a.silu, vec, pvec); break;
        default: hipLaunchKernelGGL((conv1d_fwd_kernel<T, TO, 4>), grid, block, 0, s, x, a.w, a.bias, a.pos, o, st, a.dim, a.seqlen, a.silu, vec, pvec); break;
    }
    return hipGetLastError();
}

template <typename T, typename TO, int W, bool DXF>
void conv_bwd_w(const ConvArgs& a, hipStream_t s, int vec, int pvec) {
    const ConvStates<T, TO> st{static_cast<const T*>(a.xinit), nullptr, static_cast<const T*>(a.dxfinal),
                               static_cast<TO*>(a.dxinit)};
    const unsigned nseg = (unsigned)conv_bwd_segments(a.batch, a.dim, a.seqlen);
    hipLaunchKernelGGL((conv1d_bwd_kernel<T, TO, W, kTokBwd, DXF>), dim3((unsigned)(a.batch * a.dim), nseg),
                       dim3(64), 0, s, static_cast<const T*>(a.x), a.w, a.bias, a.pos,
                       static_cast<const T*>(a.dout), static_cast<TO*>(a.out), a.partial, st, a.dim,
                       a.seqlen, a.silu, vec, pvec);
}

template <typename T, typename TO>
hipError_t conv_bwd_t(const ConvArgs& a, hipStream_t s) {
    const int vec = (a.seqlen % Storage<T>::kPerVec) == 0 && (a.seqlen % Storage<TO>::kPerVec) == 0;
    const int pvec = (a.seqlen % 4) == 0;
    const bool dxf = a.dxfinal != nullptr;
    switch (a.width) {
        case 2: dxf ? conv_bwd_w<T, TO, 2, true>(a, s, vec, pvec) : conv_bwd_w<T, TO, 2, false>(a, s, vec, pvec); break;
        case 3: dxf ? conv_bwd_w<T, TO, 3, true>(a, s, vec, pvec) : conv_bwd_w<T, TO, 3, false>(a, s, vec, pvec); break;
        default: dxf ? conv_bwd_w<T, TO, 4, true>(a, s, vec, pvec) : conv_bwd_w<T, TO, 4, false>(a, s, vec, pvec); break;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // the partials of every (batch row, segment) are summed like batch rows
    const int64_t n = a.dim * (a.width + 1);
    hipLaunchKernelGGL(conv1d_bwd_finalize, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       a.partial, a.dw, a.dbias, a.batch * conv_bwd_segments(a.batch, a.dim, a.seqlen),
                       a.dim, (int)a.width);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_conv1d_fwd(const ConvArgs& a, hipStream_t s) {
    switch (a.dtype) {
        case 1: return conv_fwd_t<bf16_t, bf16_t>(a, s);
        case 2: return conv_fwd_t<bf16_t, float>(a, s);
        default: return conv_fwd_t<float, float>(a, s);
    }
}

hipError_t launch_conv1d_bwd(const ConvArgs& a, hipStream_t s) {
    switch (a.dtype) {
        case 1: return conv_bwd_t<bf16_t, bf16_t>(a, s);
        case 2: return conv_bwd_t<bf16_t, float>(a, s);
        default: return conv_bwd_t<float, float>(a, s);
    }
}

}  // namespace pm
