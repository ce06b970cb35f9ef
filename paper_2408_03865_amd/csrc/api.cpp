// api.cpp -- the C ABI: argument validation (before anything is enqueued),
// workspace sizing and kernel launch selection.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "launch.hpp"
#include "packmamba.h"

namespace {

constexpr int64_t kMaxElems = (int64_t)1 << 40;
constexpr int kN = 16;
constexpr size_t kAlign = 256;

inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

inline bool aligned16(const void* p) { return p == nullptr || ((uintptr_t)p & 15u) == 0; }

int check_shape(int64_t batch, int64_t dim, int64_t seqlen) {
    if (batch <= 0 || dim <= 0 || seqlen <= 0) return PACKMAMBA_ERR_SHAPE;
    if (batch > 65535) return PACKMAMBA_ERR_SHAPE;                       // grid.y of the scans
    if (batch * dim > INT32_MAX) return PACKMAMBA_ERR_SHAPE;             // grid.x of the convs
    if (seqlen > INT32_MAX / 2) return PACKMAMBA_ERR_SHAPE;
    if (batch * dim > kMaxElems / seqlen) return PACKMAMBA_ERR_SHAPE;
    return PACKMAMBA_OK;
}

int check_dtype(int32_t dtype) {
    return (dtype == PACKMAMBA_F32 || dtype == PACKMAMBA_BF16 || dtype == PACKMAMBA_BF16_F32OUT)
               ? PACKMAMBA_OK
               : PACKMAMBA_ERR_UNSUPPORTED;
}

int64_t state_chunks(int64_t seqlen) {
    return (seqlen + PACKMAMBA_STATE_STRIDE - 1) / PACKMAMBA_STATE_STRIDE;
}

// Segment split workspace, shared by both directions: the per-segment maps
// (batch, dim, nseg, kN, 2) followed by the chained carries (batch, dim, nseg, kN).
// Empty when the rows are not split.
struct SegWs {
    size_t agg, carry, total;
};

SegWs seg_ws(int64_t batch, int64_t dim, int64_t seqlen, int64_t target) {
    const pm::SegPlan sp = pm::scan_segments(batch, dim, seqlen, target);
    SegWs w{0, 0, 0};
    if (sp.nseg > 1) {
        w.agg = align_up(sizeof(float) * (size_t)(batch * dim * sp.nseg * kN * 2));
        w.carry = align_up(sizeof(float) * (size_t)(batch * dim * sp.nseg * kN));
        w.total = w.agg + w.carry;
    }
    return w;
}

void set_seg_ws(pm::ScanArgs& a, char* base, const SegWs& w) {
    a.ws_agg = w.total ? reinterpret_cast<float*>(base) : nullptr;
    a.ws_carry = w.total ? reinterpret_cast<float*>(base + w.agg) : nullptr;
}

// Saved states of the forward: the chunk states (batch, dim, chunk, dstate), then the
// factor of dout in dz, fp32, per (batch, dim) row padded to whole 256-token chunks,
// each on an aligned boundary.
struct SavedLayout {
    size_t states, dzf, total;
};

SavedLayout saved_layout(int64_t batch, int64_t dim, int64_t seqlen) {
    SavedLayout s;
    s.states = align_up(sizeof(float) * (size_t)(batch * dim * state_chunks(seqlen) * kN));
    s.dzf = align_up(sizeof(float) * (size_t)(batch * dim * pm::dzf_row_len(seqlen)));
    s.total = s.states + s.dzf;
    return s;
}

// Backward workspace: dB/dC partials, per-channel partials, recomputed saved states
// (used when none are passed), then the segment workspace.
struct ScanWs {
    size_t part_bc, part_chan, states, total;
    SegWs seg;
};

ScanWs scan_ws(int64_t batch, int64_t dim, int64_t seqlen) {
    const int64_t groups = (dim + pm::kScanBwdChannels - 1) / pm::kScanBwdChannels;
    const int64_t nseg = pm::scan_segments(batch, dim, seqlen, pm::kSegTargetBwd).nseg;
    ScanWs w;
    w.part_bc = align_up(sizeof(float) * (size_t)(batch * groups * 2 * kN * seqlen));
    w.part_chan = align_up(sizeof(float) * (size_t)(batch * nseg * dim * (kN + 2)));
    w.states = saved_layout(batch, dim, seqlen).total;
    w.seg = seg_ws(batch, dim, seqlen, pm::kSegTargetBwd);   // covers the forward's plan too
    w.total = w.part_bc + w.part_chan + w.states + w.seg.total;
    return w;
}

int launch_status(hipError_t e) { return e == hipSuccess ? PACKMAMBA_OK : PACKMAMBA_ERR_LAUNCH; }

}  // namespace

namespace pm {

int conv1d_bwd_args_status(const void* x, const float* weight, const float* bias, const int32_t* position_indices,
                           const void* initial_x, const void* dout, const void* dfinal_x, const void* dx,
                           const float* dweight, const float* dbias, const void* dinitial_x, int64_t batch,
                           int64_t dim, int64_t seqlen, int32_t width, int32_t dtype) {
    if (!x || !weight || !position_indices || !dout || !dx || !dweight) return PACKMAMBA_ERR_NULL;
    if ((bias == nullptr) != (dbias == nullptr)) return PACKMAMBA_ERR_NULL;
    if ((initial_x == nullptr) != (dinitial_x == nullptr)) return PACKMAMBA_ERR_NULL;
    if (int e = check_shape(batch, dim, seqlen)) return e;
    if (int e = check_dtype(dtype)) return e;
    if (width < 2 || width > 4) return PACKMAMBA_ERR_UNSUPPORTED;
    if (!aligned16(x) || !aligned16(weight) || !aligned16(bias) || !aligned16(position_indices) ||
        !aligned16(dout) || !aligned16(dx) || !aligned16(dweight) || !aligned16(dbias) ||
        !aligned16(initial_x) || !aligned16(dfinal_x) || !aligned16(dinitial_x))
        return PACKMAMBA_ERR_ALIGN;
    return PACKMAMBA_OK;
}

int conv1d_bwd_noalloc_status(const void* x, const float* weight, const float* bias,
                              const int32_t* position_indices, const void* initial_x, const void* dout,
                              const void* dfinal_x, const void* dx, const float* dweight, const float* dbias,
                              const void* dinitial_x, int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
                              int32_t dtype) {
    if (int e = conv1d_bwd_args_status(x, weight, bias, position_indices, initial_x, dout, dfinal_x, dx, dweight,
                                       dbias, dinitial_x, batch, dim, seqlen, width, dtype))
        return e;
    if (packmamba_causal_conv1d_bwd_workspace_size(batch, dim, seqlen, width) > PACKMAMBA_NOALLOC_SCRATCH_BYTES)
        return PACKMAMBA_ERR_SCRATCH;
    return PACKMAMBA_OK;
}

}  // namespace pm

extern "C" {

int packmamba_abi_version(void) { return PACKMAMBA_ABI_VERSION; }

const char* packmamba_status_string(int status) {
    switch (status) {
        case PACKMAMBA_OK: return "ok";
        case PACKMAMBA_ERR_NULL: return "required pointer is NULL, or an optional input and its gradient disagree";
        case PACKMAMBA_ERR_SHAPE: return "invalid or too large shape";
        case PACKMAMBA_ERR_UNSUPPORTED: return "unsupported dtype, width or dstate";
        case PACKMAMBA_ERR_ALIGN: return "pointer not 16-byte aligned";
        case PACKMAMBA_ERR_WORKSPACE: return "workspace missing or too small";
        case PACKMAMBA_ERR_LAUNCH: return "kernel launch failed";
        case PACKMAMBA_ERR_SCRATCH: return "shape needs more than the fixed scratch of the no-allocation entry point";
        default: return "unknown status";
    }
}

int packmamba_causal_conv1d_fwd(const void* x, const float* weight, const float* bias,
                                const int32_t* position_indices, const void* initial_x,
                                void* out, void* final_x, int64_t batch, int64_t dim,
                                int64_t seqlen, int32_t width, int32_t dtype, int32_t silu,
                                void* stream) {
    if (!x || !weight || !position_indices || !out) return PACKMAMBA_ERR_NULL;
    if (int e = check_shape(batch, dim, seqlen)) return e;
    if (int e = check_dtype(dtype)) return e;
    if (width < 2 || width > 4) return PACKMAMBA_ERR_UNSUPPORTED;
    if (!aligned16(x) || !aligned16(weight) || !aligned16(bias) || !aligned16(position_indices) ||
        !aligned16(out) || !aligned16(initial_x) || !aligned16(final_x))
        return PACKMAMBA_ERR_ALIGN;
    pm::ConvArgs a{};
    a.x = x; a.w = weight; a.bias = bias; a.pos = position_indices; a.out = out;
    a.xinit = initial_x; a.xfinal = final_x;
    a.batch = batch; a.dim = dim; a.seqlen = seqlen; a.width = width; a.dtype = dtype;
    a.silu = silu ? 1 : 0;
    return launch_status(pm::launch_conv1d_fwd(a, (hipStream_t)stream));
}

size_t packmamba_causal_conv1d_bwd_workspace_size(int64_t batch, int64_t dim, int64_t seqlen,
                                                  int32_t width) {
    if (check_shape(batch, dim, seqlen) || width < 2 || width > 4) return 0;
    const int64_t nseg = pm::conv_bwd_segments(batch, dim, seqlen);
    return align_up(sizeof(float) * (size_t)(batch * nseg * dim * (width + 1)));
}

int packmamba_causal_conv1d_bwd(const void* x, const float* weight, const float* bias,
                                const int32_t* position_indices, const void* initial_x,
                                const void* dout, const void* dfinal_x, void* dx, float* dweight,
                                float* dbias, void* dinitial_x, void* workspace,
                                size_t workspace_bytes, int64_t batch, int64_t dim, int64_t seqlen,
                                int32_t width, int32_t dtype, int32_t silu, void* stream) {
    if (int e = pm::conv1d_bwd_args_status(x, weight, bias, position_indices, initial_x, dout, dfinal_x, dx,
                                           dweight, dbias, dinitial_x, batch, dim, seqlen, width, dtype))
        return e;
    if (!aligned16(workspace)) return PACKMAMBA_ERR_ALIGN;
    const size_t need = packmamba_causal_conv1d_bwd_workspace_size(batch, dim, seqlen, width);
    if (!workspace || workspace_bytes < need) return PACKMAMBA_ERR_WORKSPACE;
    pm::ConvArgs a{};
    a.x = x; a.w = weight; a.bias = bias; a.pos = position_indices; a.dout = dout; a.out = dx;
    a.dw = dweight; a.dbias = dbias; a.partial = static_cast<float*>(workspace);
    a.xinit = initial_x; a.dxfinal = dfinal_x; a.dxinit = dinitial_x;
    a.batch = batch; a.dim = dim; a.seqlen = seqlen; a.width = width; a.dtype = dtype;
    a.silu = silu ? 1 : 0;
    return launch_status(pm::launch_conv1d_bwd(a, (hipStream_t)stream));
}

size_t packmamba_selective_scan_fwd_saved_states_size(int64_t batch, int64_t dim, int64_t seqlen,
                                                      int32_t dstate) {
    if (check_shape(batch, dim, seqlen) || dstate != kN) return 0;
    return saved_layout(batch, dim, seqlen).total;
}

size_t packmamba_selective_scan_fwd_workspace_size(int64_t batch, int64_t dim, int64_t seqlen,
                                                   int32_t dstate) {
    if (check_shape(batch, dim, seqlen) || dstate != kN) return 0;
    return seg_ws(batch, dim, seqlen, pm::kSegTargetFwd).total;
}

int packmamba_selective_scan_fwd(const void* u, const void* delta, const float* A, const void* B,
                                 const void* C, const float* D, const void* z,
                                 const float* delta_bias, int32_t delta_softplus,
                                 const int32_t* position_indices, const float* initial_state,
                                 void* out, float* final_state, float* saved_states,
                                 void* workspace, size_t workspace_bytes, int64_t batch,
                                 int64_t dim, int64_t seqlen, int32_t dstate, int32_t dtype,
                                 void* stream) {
    if (!u || !delta || !A || !B || !C || !position_indices) return PACKMAMBA_ERR_NULL;
    if (!out && !saved_states && !final_state) return PACKMAMBA_ERR_NULL;
    if (int e = check_shape(batch, dim, seqlen)) return e;
    if (int e = check_dtype(dtype)) return e;
    if (dstate != kN) return PACKMAMBA_ERR_UNSUPPORTED;
    if (!aligned16(u) || !aligned16(delta) || !aligned16(A) || !aligned16(B) || !aligned16(C) ||
        !aligned16(D) || !aligned16(z) || !aligned16(delta_bias) ||
        !aligned16(position_indices) || !aligned16(out) || !aligned16(saved_states) ||
        !aligned16(workspace) || !aligned16(initial_state) || !aligned16(final_state))
        return PACKMAMBA_ERR_ALIGN;
    const SegWs w = seg_ws(batch, dim, seqlen, pm::kSegTargetFwd);
    if (w.total && (!workspace || workspace_bytes < w.total)) return PACKMAMBA_ERR_WORKSPACE;
    pm::ScanArgs a{};
    set_seg_ws(a, static_cast<char*>(workspace), w);
    a.u = u; a.delta = delta; a.A = A; a.B = B; a.C = C; a.D = D; a.z = z;
    a.delta_bias = delta_bias; a.pos = position_indices; a.softplus = delta_softplus ? 1 : 0;
    a.out = out; a.states = saved_states; a.h0 = initial_state; a.hfinal = final_state;
    if (saved_states && z)
        a.dzf = reinterpret_cast<float*>(reinterpret_cast<char*>(saved_states) +
                                         saved_layout(batch, dim, seqlen).states);
    a.batch = batch; a.dim = dim; a.seqlen = seqlen; a.dstate = dstate; a.dtype = dtype;
    return launch_status(pm::launch_scan_fwd(a, (hipStream_t)stream));
}

size_t packmamba_selective_scan_bwd_workspace_size(int64_t batch, int64_t dim, int64_t seqlen,
                                                   int32_t dstate) {
    if (check_shape(batch, dim, seqlen) || dstate != kN) return 0;
    return scan_ws(batch, dim, seqlen).total;
}

int packmamba_selective_scan_bwd(const void* u, const void* delta, const float* A, const void* B,
                                 const void* C, const float* D, const void* z,
                                 const float* delta_bias, int32_t delta_softplus,
                                 const int32_t* position_indices, const float* initial_state,
                                 const void* dout, const float* dfinal_state,
                                 const float* saved_states, void* du, void* ddelta, float* dA,
                                 float* dB, float* dC, float* dD, void* dz, float* ddelta_bias,
                                 float* dinitial_state,
                                 void* workspace, size_t workspace_bytes, int64_t batch,
                                 int64_t dim, int64_t seqlen, int32_t dstate, int32_t dtype,
                                 void* stream) {
    if (!u || !delta || !A || !B || !C || !position_indices || !dout) return PACKMAMBA_ERR_NULL;
    if (!du || !ddelta || !dA || !dB || !dC) return PACKMAMBA_ERR_NULL;
    if ((D == nullptr) != (dD == nullptr) || (z == nullptr) != (dz == nullptr) ||
        (delta_bias == nullptr) != (ddelta_bias == nullptr) ||
        (initial_state == nullptr) != (dinitial_state == nullptr))
        return PACKMAMBA_ERR_NULL;
    if (int e = check_shape(batch, dim, seqlen)) return e;
    if (int e = check_dtype(dtype)) return e;
    if (dstate != kN) return PACKMAMBA_ERR_UNSUPPORTED;
    const void* ptrs[] = {u, delta, A, B, C, D, z, delta_bias, position_indices, dout,
                          saved_states, du, ddelta, dA, dB, dC, dD, dz, ddelta_bias, workspace,
                          initial_state, dfinal_state, dinitial_state};
    for (const void* p : ptrs)
        if (!aligned16(p)) return PACKMAMBA_ERR_ALIGN;
    const ScanWs w = scan_ws(batch, dim, seqlen);
    if (!workspace || workspace_bytes < w.total) return PACKMAMBA_ERR_WORKSPACE;
    char* ws = static_cast<char*>(workspace);
    pm::ScanArgs a{};
    a.u = u; a.delta = delta; a.A = A; a.B = B; a.C = C; a.D = D; a.z = z;
    a.delta_bias = delta_bias; a.pos = position_indices; a.softplus = delta_softplus ? 1 : 0;
    a.batch = batch; a.dim = dim; a.seqlen = seqlen; a.dstate = dstate; a.dtype = dtype;
    a.h0 = initial_state;
    hipStream_t s = (hipStream_t)stream;
    // the forward recompute below and the backward run one after the other on the
    // stream, so they share the segment workspace
    set_seg_ws(a, ws + w.part_bc + w.part_chan + w.states, w.seg);
    char* saved = saved_states ? reinterpret_cast<char*>(const_cast<float*>(saved_states))
                               : ws + w.part_bc + w.part_chan;
    a.states = reinterpret_cast<float*>(saved);
    if (z) a.dzf = reinterpret_cast<float*>(saved + saved_layout(batch, dim, seqlen).states);
    if (!saved_states) {
        // recompute the saved states with the forward kernel (no output) into the workspace
        a.out = nullptr;
        if (int e = launch_status(pm::launch_scan_fwd(a, s))) return e;
    }
    a.dout = dout; a.du = du; a.ddelta = ddelta; a.dz = dz; a.dA = dA; a.dB = dB; a.dC = dC;
    a.dD = dD; a.ddelta_bias = ddelta_bias; a.dhfinal = dfinal_state; a.dh0 = dinitial_state;
    a.part_bc = reinterpret_cast<float*>(ws);
    a.part_chan = reinterpret_cast<float*>(ws + w.part_bc);
    return launch_status(pm::launch_scan_bwd(a, s));
}

int packmamba_rmsnorm_fwd(const void* x, const float* weight, float eps, void* out, float* rstd,
                          int64_t batch, int64_t dim, int64_t seqlen, int32_t dtype, void* stream) {
    if (!x || !weight || !out || !rstd) return PACKMAMBA_ERR_NULL;
    if (int e = check_shape(batch, dim, seqlen)) return e;
    if (int e = check_dtype(dtype)) return e;
    if (!(eps >= 0.0f)) return PACKMAMBA_ERR_SHAPE;
    if (!aligned16(x) || !aligned16(weight) || !aligned16(out) || !aligned16(rstd)) return PACKMAMBA_ERR_ALIGN;
    pm::RmsArgs a{};
    a.x = x; a.w = weight; a.out = out; a.rstd_out = rstd; a.eps = eps;
    a.batch = batch; a.dim = dim; a.seqlen = seqlen; a.dtype = dtype;
    return launch_status(pm::launch_rmsnorm_fwd(a, (hipStream_t)stream));
}

size_t packmamba_rmsnorm_bwd_workspace_size(int64_t batch, int64_t dim, int64_t seqlen) {
    if (check_shape(batch, dim, seqlen)) return 0;
    const int64_t tiles = (seqlen + pm::kRmsTile - 1) / pm::kRmsTile;
    return align_up(sizeof(float) * (size_t)((batch * tiles + pm::kRmsSlabs) * dim));
}

int packmamba_rmsnorm_bwd(const void* x, const float* weight, const float* rstd, const void* dout,
                          const void* dresidual, void* dx, float* dweight, void* workspace,
                          size_t workspace_bytes, int64_t batch, int64_t dim, int64_t seqlen,
                          int32_t dtype, void* stream) {
    if (!x || !weight || !rstd || !dout || !dx || !dweight) return PACKMAMBA_ERR_NULL;
    if (int e = check_shape(batch, dim, seqlen)) return e;
    if (int e = check_dtype(dtype)) return e;
    if (!aligned16(x) || !aligned16(weight) || !aligned16(rstd) || !aligned16(dout) ||
        !aligned16(dresidual) || !aligned16(dx) || !aligned16(dweight) || !aligned16(workspace))
        return PACKMAMBA_ERR_ALIGN;
    const size_t need = packmamba_rmsnorm_bwd_workspace_size(batch, dim, seqlen);
    if (!workspace || workspace_bytes < need) return PACKMAMBA_ERR_WORKSPACE;
    pm::RmsArgs a{};
    a.x = x; a.w = weight; a.rstd = rstd; a.dout = dout; a.dres = dresidual; a.out = dx;
    a.dw = dweight; a.partial = static_cast<float*>(workspace);
    a.batch = batch; a.dim = dim; a.seqlen = seqlen; a.dtype = dtype;
    return launch_status(pm::launch_rmsnorm_bwd(a, (hipStream_t)stream));
}

int packmamba_check_position_indices(const int32_t* position_indices, int64_t batch,
                                     int64_t seqlen, int32_t continued, int32_t* d_flag,
                                     void* stream) {
    if (!position_indices || !d_flag) return PACKMAMBA_ERR_NULL;
    if (batch <= 0 || seqlen <= 0 || batch > kMaxElems / seqlen) return PACKMAMBA_ERR_SHAPE;
    if (!aligned16(position_indices)) return PACKMAMBA_ERR_ALIGN;
    return launch_status(pm::launch_check_pos(position_indices, batch, seqlen, continued ? 1 : 0,
                                              d_flag, (hipStream_t)stream));
}

}  // extern "C"
