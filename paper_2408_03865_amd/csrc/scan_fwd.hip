// scan_fwd.hip -- packed selective scan, forward (Eqs. 1a, 1b, 2a; Alg. 2; §3.4).
//
// Layout of the work (gfx950, wave64):
//  - a block is 4 waves = 16 rows of 16 lanes; each 16-lane DPP row owns one
//    channel d of one batch row b, so a block covers 16 channels of one b;
//  - each lane owns K consecutive tokens, a row owns a chunk of 16*K tokens, and
//    the block walks the sequence chunk by chunk, carrying the state h[n] of
//    every channel from one chunk to the next in registers;
//  - B and C of the chunk (shared by the 16 channels) and the reset mask derived
//    from the position indices are staged once per chunk in LDS as fp32 with a
//    padded layout (conflict-free 16-byte reads), read from HBM with coalesced
//    vector loads (§3.5);
//  - per state n the pair (Abar, Bbar x) = (exp(dt*A), dt*B*u) is folded over the
//    lane's K tokens, the 16 lane aggregates are combined by an inclusive DPP
//    scan inside the row, the chunk carry is applied, and the lane replays its K
//    tokens from its start state to form h and y += C h.
//  - Reset (Alg. 2): Abar = exp2(dt * A*log2e + M) with M = -inf on a token whose
//    position index is 0, so the multiplier is exactly 0 there at no extra cost;
//    a product range that contains a start is therefore 0 inside the fold and the
//    scan alike (§3.4).
//  - Tokens past the row end get dt = 0 and u = 0, i.e. the identity (1, 0).
//  - When the states are saved for the backward and z is given, the kernel also
//    writes the factor (y + D u) d(z sigmoid(z))/dz of dout in dz (fp32), so that
//    the backward does not rebuild y.
//  - Long rows with few channels are split into segments scanned by different
//    blocks: an aggregate pass folds each segment into one map h -> P h + H per
//    (channel, state), a carry pass chains the maps along the row, and the main
//    pass starts each segment from its chained carry.
#include "common.hpp"
#include "launch.hpp"

namespace pm {
namespace {

constexpr int kN = 16;              // d_state
constexpr int kRows = 16;           // channels per block
constexpr int kThreads = 256;
constexpr int kStride = 128;        // saved-state token stride (PACKMAMBA_STATE_STRIDE)

template <int K>
struct __attribute__((aligned(16))) FwdSmem {
    // [state][lane][token], each lane's segment padded by 4 floats so that the
    // 16-byte reads of 8 consecutive lanes fall in distinct banks
    static constexpr int kSeg = K + 4;
    float B[kN][16][kSeg];
    float C[kN][16][kSeg];
    float M[16][kSeg];          // 0, or -inf on a sequence start
    float A2[kRows][kN];        // A * log2(e)
    float carry[kRows][kN];     // state after the previous chunk
    float pseg[kRows][kN];      // aggregate pass: product of the multipliers so far
};

struct FwdParams {
    const void* u;
    const void* delta;
    const float* A;
    const void* B;
    const void* C;
    const float* D;
    const void* z;
    const float* delta_bias;
    const int32_t* pos;
    void* out;
    float* states;
    float* dzf;               // (batch, dim, L): factor of dout in dz, or null
    const float* h0;          // state before each row (batch, dim, kN), or null
    float* hfinal;            // state after each row (batch, dim, kN), or null
    float* agg;               // aggregate pass output: (batch, dim, nseg, kN, 2) = (P, H)
    const float* carry_in;    // main pass: state before each segment (batch, dim, nseg, kN), or null
    int64_t dim, L;
    int64_t seg_chunks;       // chunks per segment
    int nseg;
    int nchunk_states;
    int softplus;
    int vec;
};

// AGG: aggregate pass over one segment (no C, no outputs), writes its map (P, H).
template <typename T, typename TO, int K, bool AGG>
__global__ __launch_bounds__(kThreads) void scan_fwd_kernel(FwdParams p) {
    constexpr int CH = 16 * K;
    constexpr int PV = Storage<T>::kPerVec;
    using Smem = FwdSmem<K>;
    __shared__ Smem sm;

    const int tid = threadIdx.x;
    const int j = tid & 15;                       // lane position inside the row
    const int r = tid >> 4;                       // row (channel) inside the block
    const int64_t b = blockIdx.y;
    const int seg = blockIdx.z;
    const int64_t d_raw = (int64_t)blockIdx.x * kRows + r;
    const bool active = d_raw < p.dim;
    const int64_t d = active ? d_raw : p.dim - 1;
    const int64_t L = p.L;
    const int64_t rowoff = (b * p.dim + d) * L;

    const T* ur = static_cast<const T*>(p.u) + rowoff;
    const T* dr = static_cast<const T*>(p.delta) + rowoff;
    const T* zr = p.z ? static_cast<const T*>(p.z) + rowoff : nullptr;
    TO* orow = p.out ? static_cast<TO*>(p.out) + rowoff : nullptr;
    const T* Bb = static_cast<const T*>(p.B) + b * kN * L;
    const T* Cb = static_cast<const T*>(p.C) + b * kN * L;
    const int32_t* pr = p.pos + b * L;

    {
        const int rr = tid >> 4, n = tid & 15;
        const int64_t dd = min((int64_t)blockIdx.x * kRows + rr, p.dim - 1);
        sm.A2[rr][n] = p.A[dd * kN + n] * kLog2e;
        float c0v = 0.0f;
        if (!AGG) {
            if (p.carry_in) c0v = p.carry_in[((b * p.dim + dd) * p.nseg + seg) * kN + n];
            else if (p.h0) c0v = p.h0[(b * p.dim + dd) * kN + n];
        }
        sm.carry[rr][n] = c0v;
        sm.pseg[rr][n] = 1.0f;
    }
    const float Dd = p.D ? p.D[d] : 0.0f;
    const float dbias = p.delta_bias ? p.delta_bias[d] : 0.0f;

    const int64_t nchunk = (L + CH - 1) / CH;
    // One chunk; FULL (block-uniform) means the chunk lies inside the row and vector
    // access is allowed, so every load and store is unconditional.
    auto chunk = [&](auto full_tag, const int64_t c) {
        constexpr bool FULL = decltype(full_tag)::value;
        const int64_t lb = c * CH;
        const int64_t l0 = lb + (int64_t)j * K;
        // this lane's inputs, loaded first in a full chunk so that their latency
        // overlaps the staging below
        RawRun<T, K> wu, wd;
        if constexpr (FULL) {
            wu = load_raw<T, K>(ur, l0);
            wd = load_raw<T, K>(dr, l0);
        }
        // ---- stage B, C and the reset mask of this chunk in LDS ----
        for (int idx = tid * PV; idx < kN * CH; idx += kThreads * PV) {
            const int n = idx / CH, t = idx - n * CH;
            float vb[PV], vc[PV];
            load_run<T, PV, FULL>(Bb + (int64_t)n * L, lb + t, L, p.vec, vb);
            if (!AGG) load_run<T, PV, FULL>(Cb + (int64_t)n * L, lb + t, L, p.vec, vc);
            float* db = &sm.B[n][t / K][t % K];
            float* dc = &sm.C[n][t / K][t % K];
#pragma unroll
            for (int q = 0; q < PV; ++q) {
                db[q] = vb[q];
                if (!AGG) dc[q] = vc[q];
            }
        }
        for (int t = tid; t < CH; t += kThreads) {
            const int64_t l = lb + t;
            sm.M[t / K][t % K] = ((FULL || l < L) && pr[l] == 0) ? -INFINITY : 0.0f;
        }
        __syncthreads();

        // ---- per-token inputs of this lane ----
        float dt[K], du[K], y[K], M[K];
        {
            float uv[K];
            if constexpr (FULL) {
                unpack_run(wu, uv);
                unpack_run(wd, dt);
            } else {
                load_run<T, K, FULL>(ur, l0, L, p.vec, uv);
                load_run<T, K, FULL>(dr, l0, L, p.vec, dt);
            }
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const float s = dt[k] + dbias;
                float v = p.softplus ? softplus_f(s) : s;
                if (!FULL) v = (l0 + k < L) ? v : 0.0f;   // identity past the row end
                dt[k] = v;
                du[k] = v * uv[k];
                y[k] = Dd * uv[k];
            }
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                const f32x4 m = *reinterpret_cast<const f32x4*>(&sm.M[j][k]);
                M[k] = m.x; M[k + 1] = m.y; M[k + 2] = m.z; M[k + 3] = m.w;
            }
        }
        // product of the lane's multipliers as one exp2 (0 if the lane holds a start)
        float S = 0.0f, Mf = 0.0f;
#pragma unroll
        for (int k = 0; k < K; ++k) { S += dt[k]; Mf += M[k]; }

        // ---- states ----
#pragma unroll 1
        for (int n = 0; n < kN; ++n) {
            // aggregate: a (channel, state) whose multiplier product is already exactly 0
            // is final; the wave skips the state when that holds for its 4 channels
            if (AGG && __all(sm.pseg[r][n] == 0.0f)) continue;
            const float A2n = sm.A2[r][n];
            const float cin = sm.carry[r][n];
            float a[K], bx[K];
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                const f32x4 bv = *reinterpret_cast<const f32x4*>(&sm.B[n][j][k]);
                const float bb[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    a[k + q] = fast_exp2(fmaf(dt[k + q], A2n, M[k + q]));
                    bx[k + q] = du[k + q] * bb[q];
                }
            }
            // fold the lane's K tokens into one affine map h -> P h + H
            float H = bx[0];
#pragma unroll
            for (int k = 1; k < K; ++k) H = fmaf(a[k], H, bx[k]);
            float P = fast_exp2(fmaf(S, A2n, Mf));
            row_scan_up(P, H);
            if (AGG) {
                // lane 15's (P, H) is the chunk's map; the chunks after it are already
                // composed in (pseg, carry), which becomes (pseg P, pseg H + carry)
                if (j == 15) {
                    const float pa = sm.pseg[r][n];
                    sm.carry[r][n] = fmaf(pa, H, sm.carry[r][n]);
                    sm.pseg[r][n] = pa * P;
                }
                continue;
            }
            const float hend = fmaf(P, cin, H);               // state after this lane's last token
            float h = dpp<kRowShr1>(cin, hend);               // state before this lane's first token
            if (j == 15) sm.carry[r][n] = hend;               // state after the chunk
#pragma unroll
            for (int k = 0; k < K; k += 4) {
                const f32x4 cv = *reinterpret_cast<const f32x4*>(&sm.C[n][j][k]);
                const float cc[4] = {cv.x, cv.y, cv.z, cv.w};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    h = fmaf(a[k + q], h, bx[k + q]);
                    y[k + q] = fmaf(cc[q], h, y[k + q]);
                }
            }
            // saved states: h after every kStride-th token
            if (p.states && active && (((j + 1) * K) % kStride) == 0) {
                const int64_t sc = (l0 + K) / kStride - 1;
                if (sc < p.nchunk_states)
                    p.states[((b * p.dim + d) * p.nchunk_states + sc) * kN + n] = hend;
            }
        }

        // ---- gate and store; for the backward, the factor of dout in dz ----
        if (!AGG && active && (orow || p.dzf)) {
            if (zr) {
                float zv[K], g[K];
                load_run<T, K, FULL>(zr, l0, L, p.vec, zv);
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    const float sz = sigmoid_f(zv[k]);
                    g[k] = y[k] * sz * (1.0f + zv[k] * (1.0f - sz));   // y d(z sigmoid(z))/dz
                    y[k] = y[k] * zv[k] * sz;
                }
                if (p.dzf) {
                    // padded row: whole vectors, also in a chunk that crosses the row end
                    float* fr = p.dzf + (b * p.dim + d) * dzf_row_len(L);
#pragma unroll
                    for (int i = 0; i < K / 4; ++i)
                        __builtin_nontemporal_store(f32x4{g[4 * i], g[4 * i + 1], g[4 * i + 2], g[4 * i + 3]},
                                                    reinterpret_cast<f32x4*>(fr + dzf_vec(c, i, j)));
                }
            }
            if (orow) store_run<TO, K, FULL>(orow, l0, L, p.vec, y);
        }
        __syncthreads();      // LDS is restaged for the next chunk
    };
    const int64_t c0 = (int64_t)seg * p.seg_chunks;
    const int64_t c1 = min(nchunk, c0 + p.seg_chunks);
    if (AGG) {
        // The aggregate composes the chunk maps from the segment's end backwards.  Once
        // the product of the multipliers is exactly 0 for every channel and state of the
        // block (a sequence start, or underflow of a long decay), the earlier chunks
        // contribute exactly nothing, and the walk stops.
        for (int64_t c = c1 - 1; c >= c0; --c) {
            if (p.vec && (c + 1) * CH <= L) chunk(std::true_type{}, c);
            else chunk(std::false_type{}, c);
            if (!__syncthreads_or(sm.pseg[tid >> 4][tid & 15] != 0.0f)) break;
        }
    } else {
        for (int64_t c = c0; c < c1; ++c) {
            if (p.vec && (c + 1) * CH <= L) chunk(std::true_type{}, c);
            else chunk(std::false_type{}, c);
        }
    }
    if (AGG) {
        __syncthreads();
        const int rr = tid >> 4, n = tid & 15;
        const int64_t dd = (int64_t)blockIdx.x * kRows + rr;
        if (dd < p.dim) {
            float* o = p.agg + (((b * p.dim + dd) * p.nseg + seg) * kN + n) * 2;
            o[0] = sm.pseg[rr][n];
            o[1] = sm.carry[rr][n];
        }
    } else if (p.hfinal && c1 == nchunk) {
        // the carry after the row's last chunk is h after its last token (tokens past
        // the row end are identities)
        const int rr = tid >> 4, n = tid & 15;
        const int64_t dd = (int64_t)blockIdx.x * kRows + rr;
        if (dd < p.dim) p.hfinal[(b * p.dim + dd) * kN + n] = sm.carry[rr][n];
    }
}

// Chains the segment maps along each row: carry[s] = state after segment s-1 (the
// row's initial state, or 0, for s = 0).
__global__ void scan_fwd_carry_kernel(const float* __restrict__ agg, float* __restrict__ carry,
                                      const float* __restrict__ h0, int64_t rows_n, int nseg) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // over batch*dim*kN
    if (i >= rows_n) return;
    const int64_t bd = i / kN;
    const int n = (int)(i - bd * kN);
    float h = h0 ? h0[i] : 0.0f;
    for (int s = 0; s < nseg; ++s) {
        const int64_t o = (bd * nseg + s) * kN + n;
        carry[o] = h;
        if (s + 1 < nseg) h = fmaf(agg[2 * o], h, agg[2 * o + 1]);
    }
}

template <typename T, typename TO, int K>
hipError_t launch_t(const ScanArgs& a, hipStream_t s) {
    static_assert(16 * K == kDzfChunk && K == 16, "the dz factor layout follows the forward's chunk");
    FwdParams p;
    p.u = a.u; p.delta = a.delta; p.A = a.A; p.B = a.B; p.C = a.C; p.D = a.D; p.z = a.z;
    p.delta_bias = a.delta_bias; p.pos = a.pos; p.out = a.out; p.states = a.states;
    p.dzf = a.z ? a.dzf : nullptr;
    p.h0 = a.h0; p.hfinal = a.hfinal;
    p.dim = a.dim; p.L = a.seqlen;
    p.nchunk_states = (int)((a.seqlen + kStride - 1) / kStride);
    p.softplus = a.softplus;
    p.vec = (a.seqlen % Storage<T>::kPerVec) == 0 && (a.seqlen % Storage<TO>::kPerVec) == 0;
    const SegPlan sp = scan_segments(a.batch, a.dim, a.seqlen, kSegTargetFwd);
    static_assert(kSegUnit % (16 * K) == 0, "segments hold whole chunks");
    p.seg_chunks = sp.seg_len / (16 * K);
    p.nseg = (int)sp.nseg;
    p.agg = a.ws_agg;
    p.carry_in = nullptr;
    const unsigned groups = (unsigned)((a.dim + kRows - 1) / kRows);
    if (sp.nseg > 1) {
        // aggregate every segment but the last, then chain
        hipLaunchKernelGGL((scan_fwd_kernel<T, TO, K, true>), dim3(groups, (unsigned)a.batch, (unsigned)(sp.nseg - 1)),
                           dim3(kThreads), 0, s, p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t rows_n = a.batch * a.dim * kN;
        hipLaunchKernelGGL(scan_fwd_carry_kernel, dim3((unsigned)((rows_n + 255) / 256)), dim3(256), 0, s,
                           a.ws_agg, a.ws_carry, a.h0, rows_n, p.nseg);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        p.carry_in = a.ws_carry;
    }
    hipLaunchKernelGGL((scan_fwd_kernel<T, TO, K, false>), dim3(groups, (unsigned)a.batch, (unsigned)sp.nseg),
                       dim3(kThreads), 0, s, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_scan_fwd(const ScanArgs& a, hipStream_t s) {
    switch (a.dtype) {
        case 1: return launch_t<bf16_t, bf16_t, 16>(a, s);
        case 2: return launch_t<bf16_t, float, 16>(a, s);
        default: return launch_t<float, float, 16>(a, s);
    }
}

}  // namespace pm
