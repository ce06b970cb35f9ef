// scan_bwd.hip -- packed selective scan, backward (§3.4), and the second-pass
// reductions of its parameter gradients.
//
// Same work layout as the forward (16-lane DPP rows = channels, K consecutive
// tokens per lane, a block = 16 channels of one batch row), with chunks of
// 16*K = 128 tokens = the saved-state stride, walked from the last to the first:
//  1. stage B, C and the reset mask of the chunk in LDS;
//  2. per state n: replay the forward inside the chunk from the saved state h at
//     the chunk start (fold, row scan, replay), keeping Abar and Abar*h_{l-1};
//  3. run the reverse recurrence dh_l = Abar_{l+1} dh_{l+1} + C_l dy_l as a
//     reverse fold + reverse DPP row scan (row_shl), entering with the carry from
//     the chunk to the right.  Abar_{l+1} of a token whose successor starts a
//     sequence is 0 (the matching reset, §3.4): it is the very Abar the replay
//     computed, shifted by one token;
//  4. accumulate du, ddelta, dz per token, dA per lane, and write the dB, dC
//     contributions; these are summed over the block's 16 channels in LDS and
//     written as one partial per block (part_bc), summed over blocks by
//     scan_bwd_finalize_bc in a fixed order.
#include "common.hpp"
#include "launch.hpp"

namespace pm {
namespace {

constexpr int kN = 16;
constexpr int kRows = 16;
constexpr int kThreads = 256;
constexpr int kK = 8;               // tokens per lane
constexpr int kCH = 16 * kK;        // tokens per chunk == saved-state stride
constexpr int kSeg = kK + 4;        // padded floats per lane segment in LDS
static_assert(kCH == 128, "chunk must equal the saved-state stride");
static_assert(kRows == kScanBwdChannels, "partials are per 16 channels");

struct BwdSmem {
    float B[kN][16][kSeg];
    float C[kN][16][kSeg];
    float M[16][kSeg];
    float red[2][2][kRows][kCH];    // [state parity][dB|dC][row][token]
};

struct BwdParams {
    const void* u;
    const void* delta;
    const float* A;
    const void* B;
    const void* C;
    const float* D;
    const void* z;
    const float* delta_bias;
    const int32_t* pos;
    const void* dout;
    const float* states;
    void* du;
    void* ddelta;
    void* dz;
    float* part_bc;       // (batch, groups, 2, kN, L)
    float* part_chan;     // (batch, dim, kN + 2): dA[n], dD, ddelta_bias
    int64_t dim, L;
    int nchunk_states;
    int groups;
    int softplus;
    int vec;
};

template <int S>
__device__ __forceinline__ void scan_step(float& P, float& H) {
    // combine with the lane S positions away (row_shr: earlier lanes; row_shl: later)
    const float Hp = dpp<S>(0.0f, H);
    const float Pp = dpp<S>(1.0f, P);
    H = fmaf(P, Hp, H);
    P = P * Pp;
}

template <typename T, typename TO>
__global__ __launch_bounds__(kThreads) void scan_bwd_kernel(BwdParams p) {
    constexpr int PV = Storage<T>::kPerVec;
    constexpr int K = kK;
    __shared__ BwdSmem sm;

    const int tid = threadIdx.x;
    const int j = tid & 15;
    const int r = tid >> 4;
    const int64_t b = blockIdx.y;
    const int64_t g = blockIdx.x;
    const int64_t d_raw = g * kRows + r;
    const bool active = d_raw < p.dim;
    const int64_t d = active ? d_raw : p.dim - 1;
    const int64_t L = p.L;
    const int64_t rowoff = (b * p.dim + d) * L;

    const T* ur = static_cast<const T*>(p.u) + rowoff;
    const T* dr = static_cast<const T*>(p.delta) + rowoff;
    const T* zr = p.z ? static_cast<const T*>(p.z) + rowoff : nullptr;
    const T* gr = static_cast<const T*>(p.dout) + rowoff;
    TO* dur = static_cast<TO*>(p.du) + rowoff;
    TO* ddr = static_cast<TO*>(p.ddelta) + rowoff;
    TO* dzr = p.dz ? static_cast<TO*>(p.dz) + rowoff : nullptr;
    const T* Bb = static_cast<const T*>(p.B) + b * kN * L;
    const T* Cb = static_cast<const T*>(p.C) + b * kN * L;
    const int32_t* pr = p.pos + b * L;
    const float* st = p.states + (b * p.dim + d) * (int64_t)p.nchunk_states * kN;

    float A2[kN], xcarry[kN], anext[kN], dAacc[kN];
#pragma unroll
    for (int n = 0; n < kN; ++n) {
        A2[n] = p.A[d * kN + n] * kLog2e;
        xcarry[n] = 0.0f;     // dh at the first token of the chunk to the right
        anext[n] = 0.0f;      // Abar at the first token of the chunk to the right
        dAacc[n] = 0.0f;
    }
    const float Dd = p.D ? p.D[d] : 0.0f;
    const float dbias = p.delta_bias ? p.delta_bias[d] : 0.0f;
    float dDacc = 0.0f, dbacc = 0.0f;

    const int64_t nchunk = (L + kCH - 1) / kCH;
    for (int64_t c = nchunk - 1; c >= 0; --c) {
        const int64_t lb = c * kCH;
        for (int idx = tid * PV; idx < kN * kCH; idx += kThreads * PV) {
            const int n = idx / kCH, t = idx - n * kCH;
            float vb[PV], vc[PV];
            load_run<T, PV>(Bb + (int64_t)n * L, lb + t, L, p.vec, vb);
            load_run<T, PV>(Cb + (int64_t)n * L, lb + t, L, p.vec, vc);
            float* db = &sm.B[n][t / K][t % K];
            float* dc = &sm.C[n][t / K][t % K];
#pragma unroll
            for (int i = 0; i < PV; ++i) { db[i] = vb[i]; dc[i] = vc[i]; }
        }
        for (int t = tid; t < kCH; t += kThreads) {
            const int64_t l = lb + t;
            sm.M[t / K][t % K] = (l < L && pr[l] == 0) ? -INFINITY : 0.0f;
        }
        __syncthreads();

        // ---- per-token inputs ----
        const int64_t l0 = lb + (int64_t)j * K;
        float uv[K], dt[K], dlu[K], dyD[K], gsp[K], M[K], yacc[K], sdhB[K], sdA[K];
        {
            float dl[K];
            load_run<T, K>(ur, l0, L, p.vec, uv);
            load_run<T, K>(dr, l0, L, p.vec, dl);
            load_run<T, K>(gr, l0, L, p.vec, dyD);     // dout for now
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const float s = dl[k] + dbias;
                float v = s;
                float gs = 1.0f;
                if (p.softplus) {
                    v = softplus_f(s);
                    gs = s > 20.0f ? 1.0f : sigmoid_f(s);
                }
                v = (l0 + k < L) ? v : 0.0f;
                dt[k] = v;
                gsp[k] = gs;
                dlu[k] = v * uv[k];
                yacc[k] = Dd * uv[k];
                sdhB[k] = 0.0f;
                sdA[k] = 0.0f;
            }
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                const f32x4 m = *reinterpret_cast<const f32x4*>(&sm.M[j][k]);
                M[k] = m.x; M[k + 1] = m.y; M[k + 2] = m.z; M[k + 3] = m.w;
            }
        }
        float zv[K];
        if (zr) {
            load_run<T, K>(zr, l0, L, p.vec, zv);
#pragma unroll
            for (int k = 0; k < K; ++k) dyD[k] *= zv[k] * sigmoid_f(zv[k]);   // dy = dout * SiLU(z)
        }

        // saved state at the chunk start (h after token lb-1)
        float hin[kN];
        if (c > 0) {
#pragma unroll
            for (int n = 0; n < kN; n += 4) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(st + (c - 1) * kN + n);
                hin[n] = v.x; hin[n + 1] = v.y; hin[n + 2] = v.z; hin[n + 3] = v.w;
            }
        } else {
#pragma unroll
            for (int n = 0; n < kN; ++n) hin[n] = 0.0f;
        }

#pragma unroll 1
        for (int n = 0; n < kN; ++n) {
            float a[K], ah[K], bv[K], cdy[K];
            float dBp[K], dCp[K];
            // ---- replay the forward inside the chunk ----
            float bx[K];
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(&sm.B[n][j][k]);
                bv[k] = v.x; bv[k + 1] = v.y; bv[k + 2] = v.z; bv[k + 3] = v.w;
            }
#pragma unroll
            for (int k = 0; k < K; ++k) {
                a[k] = fast_exp2(fmaf(dt[k], A2[n], M[k]));
                bx[k] = dlu[k] * bv[k];
            }
            float P = a[0], H = bx[0];
#pragma unroll
            for (int k = 1; k < K; ++k) {
                H = fmaf(a[k], H, bx[k]);
                P = P * a[k];
            }
            scan_step<row_shr(1)>(P, H);
            scan_step<row_shr(2)>(P, H);
            scan_step<row_shr(4)>(P, H);
            scan_step<row_shr(8)>(P, H);
            const float hend = fmaf(P, hin[n], H);
            float hprev = dpp<kRowShr1>(hin[n], hend);
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                const f32x4 cv = *reinterpret_cast<const f32x4*>(&sm.C[n][j][k]);
                const float cc[4] = {cv.x, cv.y, cv.z, cv.w};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int kk = k + q;
                    ah[kk] = a[kk] * hprev;
                    const float h = ah[kk] + bx[kk];
                    yacc[kk] = fmaf(cc[q], h, yacc[kk]);
                    dCp[kk] = dyD[kk] * h;
                    cdy[kk] = cc[q] * dyD[kk];
                    hprev = h;
                }
            }
            // ---- reverse recurrence ----
            // multiplier linking token k to k+1: a[k+1]; for the lane's last token it
            // is the next lane's a[0], or the next chunk's first token on lane 15
            const float alast = dpp<kRowShl1>(anext[n], a[0]);
            float Pr = alast, Hr = cdy[K - 1];
#pragma unroll
            for (int k = K - 2; k >= 0; --k) {
                Hr = fmaf(a[k + 1], Hr, cdy[k]);
                Pr = Pr * a[k + 1];
            }
            scan_step<row_shl(1)>(Pr, Hr);
            scan_step<row_shl(2)>(Pr, Hr);
            scan_step<row_shl(4)>(Pr, Hr);
            scan_step<row_shl(8)>(Pr, Hr);
            const float dhfirst = fmaf(Pr, xcarry[n], Hr);      // dh at this lane's first token
            float dh = dpp<kRowShl1>(xcarry[n], dhfirst);       // dh at the next lane's first token
            xcarry[n] = dpp<kNewBcast0>(0.0f, dhfirst);
            anext[n] = dpp<kNewBcast0>(0.0f, a[0]);
            float dAl = 0.0f;
#pragma unroll
            for (int k = K - 1; k >= 0; --k) {
                const float am = (k == K - 1) ? alast : a[k + 1];
                dh = fmaf(am, dh, cdy[k]);
                sdhB[k] = fmaf(dh, bv[k], sdhB[k]);
                const float q = dh * ah[k];
                sdA[k] = fmaf(q, A2[n], sdA[k]);
                dAl = fmaf(q, dt[k], dAl);
                dBp[k] = dh * dlu[k];
            }
            dAacc[n] += dAl;
            // ---- dB, dC: sum over the block's 16 channels ----
            float* rb = &sm.red[n & 1][0][r][j * K];
            float* rc = &sm.red[n & 1][1][r][j * K];
            const bool live = active;
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                f32x4 vb = {dBp[k], dBp[k + 1], dBp[k + 2], dBp[k + 3]};
                f32x4 vc = {dCp[k], dCp[k + 1], dCp[k + 2], dCp[k + 3]};
                if (!live) { vb = f32x4{0.f, 0.f, 0.f, 0.f}; vc = vb; }
                *reinterpret_cast<f32x4*>(rb + k) = vb;
                *reinterpret_cast<f32x4*>(rc + k) = vc;
            }
            __syncthreads();
            {
                const int which = tid >> 7;          // 0: dB, 1: dC
                const int t = tid & (kCH - 1);
                float s = 0.0f;
#pragma unroll
                for (int q = 0; q < kRows; ++q) s += sm.red[n & 1][which][q][t];
                const int64_t l = lb + t;
                if (l < L)
                    p.part_bc[(((b * p.groups + g) * 2 + which) * kN + n) * L + l] = s;
            }
        }

        // ---- per-token gradients ----
        float o_du[K], o_dd[K], o_dz[K];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            o_du[k] = fmaf(dyD[k], Dd, dt[k] * sdhB[k]);
            const float ddt = fmaf(uv[k], sdhB[k], sdA[k] * kLn2);   // sdA was built with A*log2e
            o_dd[k] = ddt * gsp[k];
            dDacc = fmaf(dyD[k], uv[k], dDacc);
            dbacc += (l0 + k < L) ? o_dd[k] : 0.0f;
        }
        if (zr) {
            float gv[K];
            load_run<T, K>(gr, l0, L, p.vec, gv);
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const float sz = sigmoid_f(zv[k]);
                o_dz[k] = gv[k] * yacc[k] * sz * (1.0f + zv[k] * (1.0f - sz));
            }
        }
        if (active) {
            store_run<TO, K>(dur, l0, L, p.vec, o_du);
            store_run<TO, K>(ddr, l0, L, p.vec, o_dd);
            if (dzr) store_run<TO, K>(dzr, l0, L, p.vec, o_dz);
        }
        __syncthreads();     // LDS is restaged for the next chunk
    }

    // ---- per-channel partials: sum the 16 lanes of the row ----
#pragma unroll
    for (int n = 0; n < kN; ++n) {
        float v = dAacc[n];
        v += dpp<row_shr(1)>(0.0f, v);
        v += dpp<row_shr(2)>(0.0f, v);
        v += dpp<row_shr(4)>(0.0f, v);
        v += dpp<row_shr(8)>(0.0f, v);
        dAacc[n] = v;
    }
    dDacc += dpp<row_shr(1)>(0.0f, dDacc);
    dDacc += dpp<row_shr(2)>(0.0f, dDacc);
    dDacc += dpp<row_shr(4)>(0.0f, dDacc);
    dDacc += dpp<row_shr(8)>(0.0f, dDacc);
    dbacc += dpp<row_shr(1)>(0.0f, dbacc);
    dbacc += dpp<row_shr(2)>(0.0f, dbacc);
    dbacc += dpp<row_shr(4)>(0.0f, dbacc);
    dbacc += dpp<row_shr(8)>(0.0f, dbacc);
    if (active && j == 15) {
        float* pc = p.part_chan + (b * p.dim + d) * (kN + 2);
#pragma unroll
        for (int n = 0; n < kN; ++n) pc[n] = dAacc[n];
        pc[kN] = dDacc;
        pc[kN + 1] = dbacc;
    }
}

// dB[b,n,l] / dC[b,n,l] = sum over groups of the per-block partials (fixed order)
__global__ void scan_bwd_finalize_bc(const float* __restrict__ part, float* __restrict__ dB,
                                     float* __restrict__ dC, int64_t batch, int64_t L,
                                     int groups) {
    const int64_t NL = (int64_t)kN * L;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // over batch*2*NL
    if (i >= batch * 2 * NL) return;
    const int64_t b = i / (2 * NL);
    const int64_t rem = i - b * 2 * NL;
    const int which = (int)(rem / NL);
    const int64_t nl = rem - which * NL;
    const float* src = part + ((b * groups) * 2 + which) * NL + nl;
    float s = 0.0f;
    for (int q = 0; q < groups; ++q) s += src[(int64_t)q * 2 * NL];
    (which ? dC : dB)[b * NL + nl] = s;
}

// dA[d,n], dD[d], ddelta_bias[d] = sum over batch rows (fixed order)
__global__ void scan_bwd_finalize_chan(const float* __restrict__ part, float* __restrict__ dA,
                                       float* __restrict__ dD, float* __restrict__ ddb,
                                       int64_t batch, int64_t dim) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // over dim*(kN+2)
    if (i >= dim * (kN + 2)) return;
    const int64_t d = i / (kN + 2);
    const int q = (int)(i - d * (kN + 2));
    float s = 0.0f;
    for (int64_t b = 0; b < batch; ++b) s += part[(b * dim + d) * (kN + 2) + q];
    if (q < kN) dA[d * kN + q] = s;
    else if (q == kN) { if (dD) dD[d] = s; }
    else if (ddb) ddb[d] = s;
}

template <typename T, typename TO>
hipError_t launch_t(const ScanArgs& a, hipStream_t s) {
    BwdParams p;
    p.u = a.u; p.delta = a.delta; p.A = a.A; p.B = a.B; p.C = a.C; p.D = a.D; p.z = a.z;
    p.delta_bias = a.delta_bias; p.pos = a.pos; p.dout = a.dout; p.states = a.states;
    p.du = a.du; p.ddelta = a.ddelta; p.dz = a.dz; p.part_bc = a.part_bc; p.part_chan = a.part_chan;
    p.dim = a.dim; p.L = a.seqlen;
    p.nchunk_states = (int)((a.seqlen + kCH - 1) / kCH);
    p.groups = (int)((a.dim + kRows - 1) / kRows);
    p.softplus = a.softplus;
    p.vec = (a.seqlen % Storage<T>::kPerVec) == 0 && (a.seqlen % Storage<TO>::kPerVec) == 0;
    dim3 grid((unsigned)p.groups, (unsigned)a.batch);
    hipLaunchKernelGGL((scan_bwd_kernel<T, TO>), grid, dim3(kThreads), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t nbc = a.batch * 2 * kN * a.seqlen;
    hipLaunchKernelGGL(scan_bwd_finalize_bc, dim3((unsigned)((nbc + 255) / 256)), dim3(256), 0, s,
                       a.part_bc, a.dB, a.dC, a.batch, a.seqlen, p.groups);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t nch = a.dim * (kN + 2);
    hipLaunchKernelGGL(scan_bwd_finalize_chan, dim3((unsigned)((nch + 255) / 256)), dim3(256), 0, s,
                       a.part_chan, a.dA, a.dD, a.ddelta_bias, a.batch, a.dim);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_scan_bwd(const ScanArgs& a, hipStream_t s) {
    switch (a.dtype) {
        case 1: return launch_t<bf16_t, bf16_t>(a, s);
        case 2: return launch_t<bf16_t, float>(a, s);
        default: return launch_t<float, float>(a, s);
    }
}

}  // namespace pm
