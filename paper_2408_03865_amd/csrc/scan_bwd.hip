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
//  4. accumulate du, ddelta per token, dA per lane, and write the dB, dC
//     contributions; these are summed over the block's 16 channels in LDS and
//     written as one partial per block (part_bc), summed over blocks by
//     scan_bwd_finalize_bc in a fixed order.
// dz needs y, which the forward has computed already: it saves the factor
// (y + D u) d(z sigmoid(z))/dz of dout beside the chunk states, and dz is written at
// the start of each chunk, so the state loop does not rebuild y.
// Long rows with few channels are split into segments scanned by different blocks
// (as in the forward): an aggregate pass folds each segment's reverse recurrence
// into dh_first = Q x + H, where x is dh at the first token of the next segment,
// a carry pass chains them from the row end, and the main pass enters each
// segment with its chained x.
#include "common.hpp"
#include "launch.hpp"

namespace pm {
namespace {

constexpr int kN = 16;
constexpr int kRows = 16;
constexpr int kThreads = 256;
constexpr int kK = 8;               // tokens per lane
constexpr int kCH = 16 * kK;        // tokens per chunk == saved-state stride
static_assert(kCH == 128, "chunk must equal the saved-state stride");
static_assert(kRows == kScanBwdChannels, "partials are per 16 channels");

constexpr int kWaves = kThreads / 64;
constexpr int kSeg = kK + 4;        // padded lane segment: conflict-free 16-byte LDS reads

struct __attribute__((aligned(16))) BwdSmem {
    float red[2][kWaves][2][2][kCH];   // [state parity][wave][row pair][dB|dC][token]: sums of
                                       // two channels
                                    // (first: its addresses need no constant offset)
    float B[kN][16][kSeg];          // [state][lane][token]
    float C[kN][16][kSeg];
    float M[16][kSeg];              // 0, or -inf on a sequence start
    float A2[kRows][kN];            // A * log2(e)
    float xc[kRows][kN];            // dh at the first token of the chunk to the right
    float an[kRows][kN];            // Abar at the first token of the chunk to the right
    float hin[kRows][kN];           // state at the chunk start (saved by the forward)
    float dA[kRows][kN];            // per-channel dA accumulators
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
    const float* dzf;     // (batch, dim, L): factor of dout in dz, saved by the forward
    const float* h0;      // state before each row (batch, dim, kN), or null
    const float* dhfinal; // gradient of the state after each row, or null
    float* dh0;           // gradient of h0, or null
    void* du;
    void* ddelta;
    void* dz;
    float* part_bc;       // (batch, groups, 2, kN, L)
    float* part_chan;     // (batch, nseg, dim, kN + 2): dA[n], dD, ddelta_bias
    float* agg;           // aggregate pass output: (batch, dim, nseg, kN, 2) = (Q, H)
    const float* xc_in;   // main pass: dh at the first token of the next segment, or null
    int64_t dim, L;
    int64_t seg_chunks;   // chunks per segment
    int nseg;
    int nchunk_states;
    int groups;
    int softplus;
    int vec;
};

// Step and reset mask of token l of a row (the first token after a segment), or
// (0, 0) past the row end.
template <typename T>
__device__ __forceinline__ void token_step(const T* __restrict__ dr, const int32_t* __restrict__ pr,
                                           int64_t l, int64_t L, float dbias, int softplus,
                                           float& dt, float& m) {
    dt = 0.0f;
    m = 0.0f;
    if (l < L) {
        const float s = Storage<T>::load1(dr + l) + dbias;
        dt = softplus ? softplus_f(s) : s;
        m = pr[l] == 0 ? -INFINITY : 0.0f;
    }
}

// Three waves per SIMD (at most 168 VGPRs): three blocks share a CU, so one block's
// barrier waits are covered by the other two; measured faster than two waves
// without any spill.
template <typename T, typename TO>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3, 3)))
void scan_bwd_kernel(BwdParams p) {
    constexpr int PV = Storage<T>::kPerVec;
    constexpr int K = kK;
    __shared__ BwdSmem sm;

    const int tid = threadIdx.x;
    const int j = tid & 15;
    const int r = tid >> 4;
    const int64_t b = blockIdx.y;
    const int64_t g = blockIdx.x;
    const int seg = blockIdx.z;
    const int64_t d_raw = g * kRows + r;
    const bool active = d_raw < p.dim;
    const int64_t d = active ? d_raw : p.dim - 1;
    const int64_t L = p.L;
    const int64_t rowoff = (b * p.dim + d) * L;
    const int64_t nchunk = (L + kCH - 1) / kCH;
    const int64_t c0 = (int64_t)seg * p.seg_chunks;
    const int64_t c1 = min(nchunk, c0 + p.seg_chunks);

    const T* ur = static_cast<const T*>(p.u) + rowoff;
    const T* dr = static_cast<const T*>(p.delta) + rowoff;
    const T* zr = p.z ? static_cast<const T*>(p.z) + rowoff : nullptr;
    const T* gr = static_cast<const T*>(p.dout) + rowoff;
    TO* dur = static_cast<TO*>(p.du) + rowoff;
    TO* ddr = static_cast<TO*>(p.ddelta) + rowoff;
    TO* dzr = p.dz ? static_cast<TO*>(p.dz) + rowoff : nullptr;
    const float* fr = p.dzf ? p.dzf + (b * p.dim + d) * dzf_row_len(L) : nullptr;
    const T* Bb = static_cast<const T*>(p.B) + b * kN * L;
    const T* Cb = static_cast<const T*>(p.C) + b * kN * L;
    const int32_t* pr = p.pos + b * L;

    const float Dd = p.D ? p.D[d] : 0.0f;
    const float dbias = p.delta_bias ? p.delta_bias[d] : 0.0f;
    float dDacc = 0.0f, dbacc = 0.0f;
    float dt_next, m_next;     // step and mask of the first token of the chunk to the right
    token_step<T>(dr, pr, c1 * kCH, L, dbias, p.softplus, dt_next, m_next);
    {   // per-channel tables; every lane of row rr holds the same dt_next, m_next
        const int rr = tid >> 4, n = tid & 15;
        const int64_t dd = min((int64_t)g * kRows + rr, p.dim - 1);
        const float A2n = p.A[dd * kN + n] * kLog2e;
        sm.A2[rr][n] = A2n;
        // at the row end the carry is the final state's gradient, entering h_{L-1} with
        // multiplier 1
        const bool row_end = c1 == nchunk;
        float xc0 = 0.0f;
        if (p.xc_in) xc0 = p.xc_in[((b * p.dim + dd) * p.nseg + seg) * kN + n];
        else if (row_end && p.dhfinal) xc0 = p.dhfinal[(b * p.dim + dd) * kN + n];
        sm.xc[rr][n] = xc0;
        sm.an[rr][n] = !row_end ? fast_exp2(fmaf(dt_next, A2n, m_next)) : (p.dhfinal ? 1.0f : 0.0f);
        sm.dA[rr][n] = 0.0f;
    }
    // One chunk; FULL (block-uniform) means the chunk lies inside the row and vector
    // access is allowed, so every load and store is unconditional.
    auto chunk = [&](auto full_tag, const int64_t c) {
        constexpr bool FULL = decltype(full_tag)::value;
        const int64_t lb = c * kCH;
        const int64_t l0 = lb + (int64_t)j * K;
        // this lane's inputs, loaded first in a full chunk so that their latency
        // overlaps the staging below; dout, z and the dz factor are read once
        // (non-temporal), u and delta again at the chunk end
        RawRun<T, K> wu, wd, wg, wz;
        f32x4 wf[2];
        if constexpr (FULL) {
            wu = load_raw<T, K>(ur, l0);
            wd = load_raw<T, K>(dr, l0);
            wg = load_raw_nt<T, K>(gr, l0);
            if (zr) wz = load_raw_nt<T, K>(zr, l0);
        }
        if (zr) {
            // this lane's 8 tokens of the dz factor: vectors 2 (j & 1) and 2 (j & 1) + 1 of
            // the forward's lane 8 (c & 1) + j / 2 in forward chunk c / 2 (padded row, so
            // whole vectors even past the row end)
            const int jf = 8 * (int)(c & 1) + (j >> 1), i0 = 2 * (j & 1);
            wf[0] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(fr + dzf_vec(c >> 1, i0, jf)));
            wf[1] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(fr + dzf_vec(c >> 1, i0 + 1, jf)));
        }
        // ---- stage B, C, the reset mask and the chunk-start states in LDS ----
        for (int idx = tid * PV; idx < kN * kCH; idx += kThreads * PV) {
            const int n = idx / kCH, t = idx - n * kCH;
            float vb[PV], vc[PV];
            load_run<T, PV, FULL>(Bb + (int64_t)n * L, lb + t, L, p.vec, vb);
            load_run<T, PV, FULL>(Cb + (int64_t)n * L, lb + t, L, p.vec, vc);
            float* db = &sm.B[n][t / K][t % K];
            float* dc = &sm.C[n][t / K][t % K];
#pragma unroll
            for (int i = 0; i < PV; ++i) { db[i] = vb[i]; dc[i] = vc[i]; }
        }
        for (int t = tid; t < kCH; t += kThreads) {
            const int64_t l = lb + t;
            sm.M[t / K][t % K] = ((FULL || l < L) && pr[l] == 0) ? -INFINITY : 0.0f;
        }
        {   // state at the chunk start (h after token lb-1), saved by the forward
            const int rr = tid >> 4, n = tid & 15;
            const int64_t dd = min((int64_t)g * kRows + rr, p.dim - 1);
            sm.hin[rr][n] = c > 0 ? p.states[((b * p.dim + dd) * p.nchunk_states + (c - 1)) * kN + n]
                                  : (p.h0 ? p.h0[(b * p.dim + dd) * kN + n] : 0.0f);
        }
        __syncthreads();

        // ---- per-token inputs ----
        float dt[K], dlu[K], dyD[K], sdhB[K], sdA[K];
        float S = 0.0f, Mf = 0.0f, Mr = 0.0f, m0 = 0.0f;
        {
            float dl[K], uv[K];
            if constexpr (FULL) {
                unpack_run(wu, uv);
                unpack_run(wd, dl);
                unpack_run(wg, dyD);                          // dout for now
            } else {
                load_run<T, K, FULL>(ur, l0, L, p.vec, uv);
                load_run<T, K, FULL>(dr, l0, L, p.vec, dl);
                load_run<T, K, FULL>(gr, l0, L, p.vec, dyD);
            }
            if (zr) {
                // dz = dout (y + D u) d(z sigmoid(z))/dz: the forward saved every factor
                // but dout, so dz is final here; dy = dout SiLU(z) enters the recurrence
                float zv[K];
                if constexpr (FULL) unpack_run(wz, zv);
                else load_run<T, K, FULL>(zr, l0, L, p.vec, zv);
                float fz[K] = {wf[0].x, wf[0].y, wf[0].z, wf[0].w, wf[1].x, wf[1].y, wf[1].z, wf[1].w};
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    fz[k] *= dyD[k];
                    dyD[k] *= zv[k] * sigmoid_f(zv[k]);
                }
                if (active) store_run<TO, K, FULL, true>(dzr, l0, L, p.vec, fz);
            }
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const float s = dl[k] + dbias;
                float v = s;
                if (p.softplus) v = softplus_f(s);
                if (!FULL) v = (l0 + k < L) ? v : 0.0f;   // identity past the row end
                dt[k] = v;
                if (!active) dyD[k] = 0.0f;           // padding rows contribute nothing to dB, dC
                dlu[k] = active ? v * uv[k] : 0.0f;
                dDacc = fmaf(dyD[k], uv[k], dDacc);
                sdhB[k] = 0.0f;
                sdA[k] = 0.0f;
            }
            // Lane products of Abar as one exp2 each: prod_k exp2(dt_k A2) = exp2(A2 sum_k dt_k),
            // forced to 0 when a reset falls inside the product range.
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                const f32x4 m = *reinterpret_cast<const f32x4*>(&sm.M[j][k]);
                const float mm[4] = {m.x, m.y, m.z, m.w};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    S += dt[k + q];
                    Mf += mm[q];
                    if (k + q > 0) Mr += mm[q];
                }
                if (k == 0) m0 = mm[0];
            }
        }
        const float dt0n = dpp<kRowShl1>(dt_next, dt[0]);    // next token's step, across the lane edge
        const float m0n = dpp<kRowShl1>(m_next, m0);
        const float Sr = S - dt[0] + dt0n;
        Mr += m0n;
        dt_next = dpp<kNewBcast0>(0.0f, dt[0]);
        m_next = dpp<kNewBcast0>(0.0f, m0);

        // per-thread LDS addresses of the dB/dC sums and the offset of this thread's
        // partial (token red_t of dB or dC) inside the block's state-0 partials
        const int wr = r & 3;                        // row inside the wave
        float* const red_w = &sm.red[0][tid >> 6][wr & 1][wr >> 1][j * K];
        const int red_which = __builtin_amdgcn_readfirstlane(tid >> 7);   // 0: dB, 1: dC (per wave)
        const int red_t = tid & (kCH - 1);
        const float* const red_r = &sm.red[0][0][0][red_which][red_t];
        float* const part_n = p.part_bc + ((b * p.groups + g) * 2 + red_which) * kN * L;
        const uint32_t part_off = (uint32_t)(lb + red_t);
#pragma unroll 1
        for (int n = 0; n < kN; ++n) {
            const float A2n = sm.A2[r][n];
            const float hin = sm.hin[r][n];
            const float xc = sm.xc[r][n];
            const float an = sm.an[r][n];
            float a[K], ah[K], bv[K], cdy[K], bx[K], M[K];
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                const f32x4 m = *reinterpret_cast<const f32x4*>(&sm.M[j][k]);
                M[k] = m.x; M[k + 1] = m.y; M[k + 2] = m.z; M[k + 3] = m.w;
            }
            // ---- fold the lane's tokens both ways, then both row scans at once ----
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(&sm.B[n][j][k]);
                bv[k] = v.x; bv[k + 1] = v.y; bv[k + 2] = v.z; bv[k + 3] = v.w;
                const f32x4 cv = *reinterpret_cast<const f32x4*>(&sm.C[n][j][k]);
                cdy[k] = cv.x * dyD[k]; cdy[k + 1] = cv.y * dyD[k + 1];
                cdy[k + 2] = cv.z * dyD[k + 2]; cdy[k + 3] = cv.w * dyD[k + 3];
            }
#pragma unroll
            for (int k = 0; k < K; ++k) {
                a[k] = fast_exp2(fmaf(dt[k], A2n, M[k]));
                bx[k] = dlu[k] * bv[k];
            }
            // forward: h -> P h + H over the lane's tokens
            float H = bx[0];
#pragma unroll
            for (int k = 1; k < K; ++k) H = fmaf(a[k], H, bx[k]);
            // reverse: dh_l = Abar_{l+1} dh_{l+1} + C_l dy_l over the lane's tokens
            float Hr = cdy[K - 1];
#pragma unroll
            for (int k = K - 2; k >= 0; --k) Hr = fmaf(a[k + 1], Hr, cdy[k]);
            float P = fast_exp2(fmaf(S, A2n, Mf));
            float Pr = fast_exp2(fmaf(Sr, A2n, Mr));
            // Wave priority (s_setprio, per wave, relative to the other waves of the SIMD):
            // raised over this DPP latency chain, and from the reverse recurrence to the
            // state's barrier, so that the block's waves reach the barrier sooner; the
            // other blocks' waves fill the issue slots meanwhile (-4% at 8 x 4096 x 4096).
            __builtin_amdgcn_s_setprio(1);
            row_scan_up_down(P, H, Pr, Hr);
            __builtin_amdgcn_s_setprio(0);
            // ---- replay the forward inside the chunk ----
            const float hend = fmaf(P, hin, H);
            float hprev = dpp<kRowShr1>(hin, hend);
#pragma unroll
            for (int k = 0; k < K; ++k) {
                ah[k] = a[k] * hprev;
                const float h = ah[k] + bx[k];
                bx[k] = dyD[k] * h;                          // dC contribution (reuses bx)
                hprev = h;
            }
            // ---- reverse recurrence, entering with the carry from the right ----
            const float alast = dpp<kRowShl1>(an, a[0]);        // Abar of the next lane's first token
            const float dhfirst = fmaf(Pr, xc, Hr);            // dh at this lane's first token
            float dh = dpp<kRowShl1>(xc, dhfirst);               // dh at the next lane's first token
            if (j == 0) {
                sm.xc[r][n] = dhfirst;
                sm.an[r][n] = a[0];
            }
            __builtin_amdgcn_s_setprio(2);
            float dAl = 0.0f;
            float dBp[K];
#pragma unroll
            for (int k = K - 1; k >= 0; --k) {
                const float am = (k == K - 1) ? alast : a[k + 1];
                dh = fmaf(am, dh, cdy[k]);
                sdhB[k] = fmaf(dh, bv[k], sdhB[k]);
                const float q = dh * ah[k];
                sdA[k] = fmaf(q, A2n, sdA[k]);
                dAl = fmaf(q, dt[k], dAl);
                dBp[k] = dh * dlu[k];
            }
            dAl = row_sum_to_15(dAl);
            if (j == 15) sm.dA[r][n] += dAl;
            // ---- dB, dC: sum over the block's 16 channels ----
            // First over pairs of the wave's 4 rows (channels) in registers:
            // permlane32_swap pairs rows {0,1} with {2,3} and leaves dB sums on rows 0-1
            // and dC sums on rows 2-3 (one swap and one add per pair of values; a second
            // swap stage over even and odd rows measured slower than summing eight
            // partials instead of four from LDS).
            float R[K];
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const auto s2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(dBp[k]),
                                                                 __float_as_uint(bx[k]), false, false);
                R[k] = __uint_as_float(s2[0]) + __uint_as_float(s2[1]);
            }
            const int par = (n & 1) * (kWaves * 4 * kCH);
            *reinterpret_cast<f32x4*>(red_w + par) = f32x4{R[0], R[1], R[2], R[3]};
            *reinterpret_cast<f32x4*>(red_w + par + 4) = f32x4{R[4], R[5], R[6], R[7]};
            __syncthreads();
            __builtin_amdgcn_s_setprio(0);
            {   // then over the block's 4 waves x 2 row pairs, in a fixed order
                float s = 0.0f;
#pragma unroll
                for (int q = 0; q < 2 * kWaves; ++q) s += red_r[par + q * 2 * kCH];
                if (FULL || lb + red_t < L) __builtin_nontemporal_store(s, &part_n[n * L + part_off]);   // read once, by the finalize
            }
            // no second barrier: the next state writes the other buffer, and this one is
            // rewritten only after every thread has passed the next state's barrier
        }

        // ---- per-token gradients ----
        float o_du[K], o_dd[K];
        {
            float uv[K], dl[K];
            load_run<T, K, FULL>(ur, l0, L, p.vec, uv);
            load_run<T, K, FULL>(dr, l0, L, p.vec, dl);
#pragma unroll
            for (int k = 0; k < K; ++k) {
                o_du[k] = fmaf(dyD[k], Dd, dt[k] * sdhB[k]);
                const float ddt = fmaf(uv[k], sdhB[k], sdA[k] * kLn2);   // sdA was built with A*log2e
                const float s = dl[k] + dbias;
                o_dd[k] = p.softplus ? ddt * softplus_grad_f(s, dt[k]) : ddt;
                dbacc += (FULL || l0 + k < L) ? o_dd[k] : 0.0f;
            }
        }
        if (active) {
            store_run<TO, K, FULL, true>(dur, l0, L, p.vec, o_du);
            store_run<TO, K, FULL, true>(ddr, l0, L, p.vec, o_dd);
        }
        __syncthreads();     // LDS is restaged for the next chunk
    };
    for (int64_t c = c1 - 1; c >= c0; --c) {
        if (p.vec && (c + 1) * kCH <= L) chunk(std::true_type{}, c);
        else chunk(std::false_type{}, c);
    }

    // ---- per-channel partials ----
    dDacc = row_sum_to_15(dDacc);
    dbacc = row_sum_to_15(dbacc);
    // gradient of the initial state: dh at token 0 times Abar at token 0 (0 at a start),
    // both left in LDS by lane 0 after the first chunk
    if (p.dh0 && c0 == 0) {
        const int rr = tid >> 4, n = tid & 15;
        const int64_t dd = g * kRows + rr;
        if (dd < p.dim) p.dh0[(b * p.dim + dd) * kN + n] = sm.an[rr][n] * sm.xc[rr][n];
    }
    float* pcb = p.part_chan + (b * p.nseg + seg) * p.dim * (kN + 2);
    if (active && j == 15) {
        float* pc = pcb + d * (kN + 2);
        pc[kN] = dDacc;
        pc[kN + 1] = dbacc;
    }
    {
        const int rr = tid >> 4, n = tid & 15;
        if ((int64_t)g * kRows + rr < p.dim)
            pcb[(g * kRows + rr) * (kN + 2) + n] = sm.dA[rr][n];
    }
}

// Aggregate pass of one segment (blockIdx.z + 1; the first segment needs none): the
// reverse recurrence over the segment with x = 0 gives H = dh at its first token,
// and Q = the product of the multipliers Abar_{l+1} over its tokens l, so that
// dh_first = Q x + H.  Same arithmetic as the main pass, without the forward replay
// and the gradients.
struct __attribute__((aligned(16))) AggSmem {
    float C[kN][16][kSeg];
    float M[16][kSeg];
    float A2[kRows][kN];
    float xc[kRows][kN];
    float q[kRows][kN];
};

template <typename T>
__global__ __launch_bounds__(kThreads) void scan_bwd_agg_kernel(BwdParams p) {
    constexpr int PV = Storage<T>::kPerVec;
    constexpr int K = kK;
    __shared__ AggSmem sm;

    const int tid = threadIdx.x;
    const int j = tid & 15;
    const int r = tid >> 4;
    const int64_t b = blockIdx.y;
    const int64_t g = blockIdx.x;
    const int seg = blockIdx.z + 1;
    const int64_t d = min(g * kRows + r, p.dim - 1);
    const int64_t L = p.L;
    const int64_t rowoff = (b * p.dim + d) * L;
    const int64_t nchunk = (L + kCH - 1) / kCH;
    const int64_t c0 = (int64_t)seg * p.seg_chunks;
    const int64_t c1 = min(nchunk, c0 + p.seg_chunks);

    const T* dr = static_cast<const T*>(p.delta) + rowoff;
    const T* zr = p.z ? static_cast<const T*>(p.z) + rowoff : nullptr;
    const T* gr = static_cast<const T*>(p.dout) + rowoff;
    const T* Cb = static_cast<const T*>(p.C) + b * kN * L;
    const int32_t* pr = p.pos + b * L;

    const float dbias = p.delta_bias ? p.delta_bias[d] : 0.0f;
    {
        const int rr = tid >> 4, n = tid & 15;
        const int64_t dd = min(g * kRows + rr, p.dim - 1);
        sm.A2[rr][n] = p.A[dd * kN + n] * kLog2e;
        sm.xc[rr][n] = 0.0f;
        sm.q[rr][n] = 1.0f;
    }

    auto chunk = [&](auto full_tag, const int64_t c) {
        constexpr bool FULL = decltype(full_tag)::value;
        const int64_t lb = c * kCH;
        float dt_next, m_next;     // step and mask of the first token after the chunk
        token_step<T>(dr, pr, lb + kCH, L, dbias, p.softplus, dt_next, m_next);
        for (int idx = tid * PV; idx < kN * kCH; idx += kThreads * PV) {
            const int n = idx / kCH, t = idx - n * kCH;
            float vc[PV];
            load_run<T, PV, FULL>(Cb + (int64_t)n * L, lb + t, L, p.vec, vc);
            float* dc = &sm.C[n][t / K][t % K];
#pragma unroll
            for (int i = 0; i < PV; ++i) dc[i] = vc[i];
        }
        for (int t = tid; t < kCH; t += kThreads) {
            const int64_t l = lb + t;
            sm.M[t / K][t % K] = ((FULL || l < L) && pr[l] == 0) ? -INFINITY : 0.0f;
        }
        __syncthreads();

        const int64_t l0 = lb + (int64_t)j * K;
        float dt[K], dyD[K], M[K];
        float S = 0.0f, Mr = 0.0f;
        {
            float dl[K];
            load_run<T, K, FULL>(dr, l0, L, p.vec, dl);
            load_run<T, K, FULL>(gr, l0, L, p.vec, dyD);
            if (zr) {
                float zv[K];
                load_run<T, K, FULL>(zr, l0, L, p.vec, zv);
#pragma unroll
                for (int k = 0; k < K; ++k) dyD[k] *= zv[k] * sigmoid_f(zv[k]);
            }
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const float s = dl[k] + dbias;
                float v = s;
                if (p.softplus) v = softplus_f(s);
                if (!FULL) v = (l0 + k < L) ? v : 0.0f;
                dt[k] = v;
            }
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                const f32x4 m = *reinterpret_cast<const f32x4*>(&sm.M[j][k]);
                M[k] = m.x; M[k + 1] = m.y; M[k + 2] = m.z; M[k + 3] = m.w;
            }
#pragma unroll
            for (int k = 0; k < K; ++k) {
                S += dt[k];
                if (k > 0) Mr += M[k];
            }
        }
        const float dt0n = dpp<kRowShl1>(dt_next, dt[0]);
        const float m0n = dpp<kRowShl1>(m_next, M[0]);
        const float Sr = S - dt[0] + dt0n;
        Mr += m0n;

#pragma unroll 1
        for (int n = 0; n < kN; ++n) {
            // a (channel, state) whose multiplier product is already exactly 0 is final;
            // the wave skips the state when that holds for its 4 channels
            if (__all(sm.q[r][n] == 0.0f)) continue;
            const float A2n = sm.A2[r][n];
            float cdy[K];
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                const f32x4 cv = *reinterpret_cast<const f32x4*>(&sm.C[n][j][k]);
                cdy[k] = cv.x * dyD[k]; cdy[k + 1] = cv.y * dyD[k + 1];
                cdy[k + 2] = cv.z * dyD[k + 2]; cdy[k + 3] = cv.w * dyD[k + 3];
            }
            float Hr = cdy[K - 1];
#pragma unroll
            for (int k = K - 2; k >= 0; --k)
                Hr = fmaf(fast_exp2(fmaf(dt[k + 1], A2n, M[k + 1])), Hr, cdy[k]);
            float Pr = fast_exp2(fmaf(Sr, A2n, Mr));
            row_scan_down(Pr, Hr);
            // lane 0's (Pr, Hr) is the chunk's map from dh after the chunk to dh at its
            // first token; the chunks before it are already composed in (q, xc), which
            // becomes (q Pr, q Hr + xc)
            if (j == 0) {
                const float qa = sm.q[r][n];
                sm.xc[r][n] = fmaf(qa, Hr, sm.xc[r][n]);
                sm.q[r][n] = qa * Pr;
            }
        }
        __syncthreads();
    };
    // The chunk maps are composed from the segment's start forwards.  Once the product
    // of the multipliers is exactly 0 for every channel and state of the block (the
    // token before a sequence start, or underflow of a long decay), the later chunks
    // contribute exactly nothing, and the walk stops.
    for (int64_t c = c0; c < c1; ++c) {
        if (p.vec && (c + 1) * kCH <= L) chunk(std::true_type{}, c);
        else chunk(std::false_type{}, c);
        if (!__syncthreads_or(sm.q[tid >> 4][tid & 15] != 0.0f)) break;
    }
    {
        const int rr = tid >> 4, n = tid & 15;
        const int64_t dd = g * kRows + rr;
        if (dd < p.dim) {
            float* o = p.agg + (((b * p.dim + dd) * p.nseg + seg) * kN + n) * 2;
            o[0] = sm.q[rr][n];
            o[1] = sm.xc[rr][n];
        }
    }
}

// Chains the segment maps from the row end: xc[s] = dh at the first token of segment
// s+1 (the final state's gradient, or 0, for the last segment).
__global__ void scan_bwd_carry_kernel(const float* __restrict__ agg, float* __restrict__ xc,
                                      const float* __restrict__ dhfinal, int64_t rows_n, int nseg) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // over batch*dim*kN
    if (i >= rows_n) return;
    const int64_t bd = i / kN;
    const int n = (int)(i - bd * kN);
    float x = dhfinal ? dhfinal[i] : 0.0f;
    for (int s = nseg - 1; s >= 0; --s) {
        const int64_t o = (bd * nseg + s) * kN + n;
        xc[o] = x;
        if (s > 0) x = fmaf(agg[2 * o], x, agg[2 * o + 1]);
    }
}

// dB[b,n,l] / dC[b,n,l] = sum over groups of the per-block partials.  Each thread owns
// four consecutive tokens and keeps four running sums over interleaved groups
// (q mod 4), added at the end: a fixed order, so the result is reproducible.
__global__ void scan_bwd_finalize_bc(const float* __restrict__ part, float* __restrict__ dB,
                                     float* __restrict__ dC, int64_t batch, int64_t L,
                                     int groups) {
    const int64_t NL = (int64_t)kN * L;
    const int64_t i4 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;   // over batch*2*NL
    if (i4 >= batch * 2 * NL) return;
    const int64_t b = i4 / (2 * NL);
    const int64_t rem = i4 - b * 2 * NL;
    const int which = (int)(rem / NL);
    const int64_t nl = rem - which * NL;
    const float* src = part + ((b * groups) * 2 + which) * NL + nl;
    const int64_t stride = 2 * NL;
    float* dst = (which ? dC : dB) + b * NL + nl;
    // NL = 16 L, so a group of four never crosses a (b, dB|dC) boundary and every
    // offset is a multiple of four floats (16-byte aligned).
    f32x4 acc[4] = {};
    int q = 0;
    for (; q + 4 <= groups; q += 4) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            acc[u] += *reinterpret_cast<const f32x4*>(src + (int64_t)(q + u) * stride);
    }
    for (; q < groups; ++q) acc[q & 3] += *reinterpret_cast<const f32x4*>(src + (int64_t)q * stride);
    *reinterpret_cast<f32x4*>(dst) = (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

// dA[d,n], dD[d], ddelta_bias[d] = sum over batch rows and segments (fixed order)
__global__ void scan_bwd_finalize_chan(const float* __restrict__ part, float* __restrict__ dA,
                                       float* __restrict__ dD, float* __restrict__ ddb,
                                       int64_t nparts, int64_t dim) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // over dim*(kN+2)
    if (i >= dim * (kN + 2)) return;
    const int64_t d = i / (kN + 2);
    const int q = (int)(i - d * (kN + 2));
    float s = 0.0f;
    for (int64_t b = 0; b < nparts; ++b) s += part[(b * dim + d) * (kN + 2) + q];
    if (q < kN) dA[d * kN + q] = s;
    else if (q == kN) { if (dD) dD[d] = s; }
    else if (ddb) ddb[d] = s;
}

template <typename T, typename TO>
hipError_t launch_t(const ScanArgs& a, hipStream_t s) {
    static_assert(kK == 8 && 2 * kCH == kDzfChunk, "the dz factor layout follows the forward's chunk");
    BwdParams p;
    p.u = a.u; p.delta = a.delta; p.A = a.A; p.B = a.B; p.C = a.C; p.D = a.D; p.z = a.z;
    p.delta_bias = a.delta_bias; p.pos = a.pos; p.dout = a.dout; p.states = a.states;
    p.dzf = a.z ? a.dzf : nullptr;
    if (a.z && !a.dzf) return hipErrorInvalidValue;
    p.h0 = a.h0; p.dhfinal = a.dhfinal; p.dh0 = a.dh0;
    p.du = a.du; p.ddelta = a.ddelta; p.dz = a.dz; p.part_bc = a.part_bc; p.part_chan = a.part_chan;
    p.dim = a.dim; p.L = a.seqlen;
    p.nchunk_states = (int)((a.seqlen + kCH - 1) / kCH);
    p.groups = (int)((a.dim + kRows - 1) / kRows);
    p.softplus = a.softplus;
    p.vec = (a.seqlen % Storage<T>::kPerVec) == 0 && (a.seqlen % Storage<TO>::kPerVec) == 0;
    const SegPlan sp = scan_segments(a.batch, a.dim, a.seqlen, kSegTargetBwd);
    static_assert(kSegUnit % kCH == 0, "segments hold whole chunks");
    p.seg_chunks = sp.seg_len / kCH;
    p.nseg = (int)sp.nseg;
    p.agg = a.ws_agg;
    p.xc_in = nullptr;
    hipError_t e;
    if (sp.nseg > 1) {
        hipLaunchKernelGGL((scan_bwd_agg_kernel<T>), dim3((unsigned)p.groups, (unsigned)a.batch, (unsigned)(sp.nseg - 1)),
                           dim3(kThreads), 0, s, p);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t rows_n = a.batch * a.dim * kN;
        hipLaunchKernelGGL(scan_bwd_carry_kernel, dim3((unsigned)((rows_n + 255) / 256)), dim3(256), 0, s,
                           a.ws_agg, a.ws_carry, a.dhfinal, rows_n, p.nseg);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        p.xc_in = a.ws_carry;
    }
    hipLaunchKernelGGL((scan_bwd_kernel<T, TO>), dim3((unsigned)p.groups, (unsigned)a.batch, (unsigned)sp.nseg),
                       dim3(kThreads), 0, s, p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t nbc4 = (a.batch * 2 * kN * a.seqlen + 3) / 4;
    hipLaunchKernelGGL(scan_bwd_finalize_bc, dim3((unsigned)((nbc4 + 255) / 256)), dim3(256), 0, s,
                       a.part_bc, a.dB, a.dC, a.batch, a.seqlen, p.groups);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t nch = a.dim * (kN + 2);
    hipLaunchKernelGGL(scan_bwd_finalize_chan, dim3((unsigned)((nch + 255) / 256)), dim3(256), 0, s,
                       a.part_chan, a.dA, a.dD, a.ddelta_bias, a.batch * sp.nseg, a.dim);
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
