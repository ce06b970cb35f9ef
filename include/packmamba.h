/*
 * packmamba.h -- C ABI of the packed causal conv1d and packed selective scan
 * (PackMamba, arXiv 2408.03865) on AMD Instinct MI355X (gfx950).
 *
 * Packing (§3.1): many variable-length sequences are concatenated along the
 * sequence axis into rows of length `seqlen`; `position_indices` (batch, seqlen)
 * int32 holds each token's 0-based position inside its own sequence, so a 0
 * marks a sequence start.  Neither operator passes information across a start:
 * the conv drops taps that reach before the start (Alg. 1, §3.3) and the scan
 * forces its multiplier exp(delta * A) to 0 at the start (Alg. 2, §3.4).
 *
 * Conventions shared by every entry point
 *  - Every pointer is a DEVICE pointer owned by the caller.  The library never
 *    allocates, frees or synchronises; it only enqueues kernels on `stream`
 *    (a hipStream_t; NULL means the null stream).  It keeps no mutable global
 *    state, so concurrent calls on different streams are independent -- except
 *    packmamba_causal_conv1d_bwd_noalloc, whose fixed scratch buffer is shared by
 *    every call on a device (see there).
 *  - Layout: contiguous, row-major, sequence axis innermost:
 *      activations (x, u, delta, z, out, dout and their gradients)  (batch, dim, seqlen)
 *      B, C, dB, dC                                                 (batch, dstate, seqlen)
 *      A, dA                                                        (dim, dstate)
 *      conv weight and dweight                                      (dim, width)
 *      D, delta_bias, conv bias and their gradients                 (dim)
 *      position_indices                                             (batch, seqlen)
 *  - dtype: activation inputs (x, u, delta, z, dout), B and C are float
 *    (PACKMAMBA_F32) or bfloat16 bits (PACKMAMBA_BF16, PACKMAMBA_BF16_F32OUT).
 *    Activation outputs (out, dx, du, ddelta, dz) are bfloat16 for
 *    PACKMAMBA_BF16 and float otherwise.  Parameters, their gradients, dB and dC
 *    are always float.  Arithmetic and scan state are fp32; bfloat16 outputs
 *    are rounded once, to nearest even.
 *  - Every pointer must be 16-byte aligned (PACKMAMBA_ERR_ALIGN otherwise).
 *  - Argument errors are returned synchronously, before anything is enqueued.
 *    Faults inside kernels are asynchronous and surface at the caller's next
 *    synchronisation.  PACKMAMBA_ERR_LAUNCH reports a failed launch.
 *  - Precondition (not checked on the hot path): position_indices[b,0] == 0 and
 *    position_indices[b,l] is 0 or position_indices[b,l-1]+1.
 *    packmamba_check_position_indices() verifies it on demand.
 *  - State passing across rows (the future work of §5: a long sequence cut at a
 *    row end continues in another row).  Every operator takes optional per-row
 *    initial states and returns final states, with their gradients.  A row that
 *    continues a sequence has its first position index equal to that token's
 *    position in the sequence (then any value >= 0); a 0 there starts a new
 *    sequence and cuts the initial state off, as any start does.  Passing a
 *    row's final states as the next part's initial states makes the two parts
 *    compute exactly what the uncut row computes; without initial states a
 *    continued sequence sees zeros.  All state pointers may be NULL.
 */
#ifndef PACKMAMBA_H
#define PACKMAMBA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PACKMAMBA_ABI_VERSION 6

/* dtype codes of the activation tensors */
#define PACKMAMBA_F32 0            /* fp32 inputs, fp32 outputs */
#define PACKMAMBA_BF16 1           /* bf16 inputs, bf16 outputs */
#define PACKMAMBA_BF16_F32OUT 2    /* bf16 inputs, fp32 outputs (same arithmetic as PACKMAMBA_BF16,
                                      before the final rounding) */

/* Token stride of the scan states saved by the forward for the backward. */
#define PACKMAMBA_STATE_STRIDE 128

typedef enum {
    PACKMAMBA_OK = 0,
    PACKMAMBA_ERR_NULL = 1,         /* required pointer NULL, or a gradient/optional-input pair mismatched */
    PACKMAMBA_ERR_SHAPE = 2,        /* a dimension <= 0, or sizes overflow */
    PACKMAMBA_ERR_UNSUPPORTED = 3,  /* dtype, width (2..4) or dstate (16) not supported */
    PACKMAMBA_ERR_ALIGN = 4,        /* a pointer is not 16-byte aligned */
    PACKMAMBA_ERR_WORKSPACE = 5,    /* workspace NULL or smaller than the *_workspace_size() result */
    PACKMAMBA_ERR_LAUNCH = 6,       /* the HIP runtime rejected a kernel launch */
    PACKMAMBA_ERR_SCRATCH = 7       /* the shape needs more than the fixed scratch of a no-allocation entry point */
} packmamba_status;

/* ABI version of the loaded library (PACKMAMBA_ABI_VERSION). */
int packmamba_abi_version(void);

/* Static, NUL-terminated description of a status code. */
const char* packmamba_status_string(int status);

/*
 * Causal depthwise conv1d with sequence-start masking, forward (Alg. 1, §3.3).
 *   pre[b,d,l] = bias[d] + sum_{k=0}^{width-1} [k <= pos[b,l]] * weight[d,width-1-k] * x[b,d,l-k]
 *   out = silu ? pre * sigmoid(pre) : pre
 * The tap that reaches k tokens back is used only if it stays inside the output
 * token's own sequence; weight[d, width-1] multiplies the current token.  A tap
 * reaching before the row (a continued sequence) reads initial_x.
 *   x, out: dtype (batch, dim, seqlen); weight (dim, width); bias (dim) or NULL;
 *   width in [2, 4].
 *   initial_x: NULL, or (batch, dim, width-1) in x's storage type: the inputs of
 *   the width-1 tokens before each row, token -1 last (NULL reads zeros).
 *   final_x: NULL, or (batch, dim, width-1) in x's storage type, receives each
 *   row's last width-1 inputs, copied (from initial_x where the row is shorter).
 */
int packmamba_causal_conv1d_fwd(const void* x, const float* weight, const float* bias,
                                const int32_t* position_indices, const void* initial_x,
                                void* out, void* final_x,
                                int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
                                int32_t dtype, int32_t silu, void* stream);

/* Bytes of workspace packmamba_causal_conv1d_bwd needs. */
size_t packmamba_causal_conv1d_bwd_workspace_size(int64_t batch, int64_t dim, int64_t seqlen,
                                                  int32_t width);

/*
 * Causal conv1d backward (§3.3, §3.5): gradients of sum(dout * out).
 *   dx[b,d,j] = sum_k [pos[b,j+k] >= k] * weight[d,width-1-k] * g[b,d,j+k]
 *   (the "reverse indices" of the next width-1 tokens), with g = dout * d out/d pre;
 *   dweight[d,width-1-k] = sum_{b,l} [k <= pos[b,l]] g[b,d,l] x[b,d,l-k];
 *   dbias[d] = sum_{b,l} g[b,d,l].
 *   dx: dtype; dweight (dim, width) and dbias (dim) are overwritten; dbias must
 *   be NULL iff bias is NULL.  The parameter sums are deterministic (fixed order).
 *   initial_x: as in the forward.  dfinal_x: NULL (zero), or the gradient of
 *   final_x, (batch, dim, width-1) in dout's storage type.  dinitial_x: the
 *   gradient of initial_x, (batch, dim, width-1) in dx's type; it must be NULL iff
 *   initial_x is NULL.
 */
int packmamba_causal_conv1d_bwd(const void* x, const float* weight, const float* bias,
                                const int32_t* position_indices, const void* initial_x,
                                const void* dout, const void* dfinal_x,
                                void* dx, float* dweight, float* dbias, void* dinitial_x,
                                void* workspace, size_t workspace_bytes,
                                int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
                                int32_t dtype, int32_t silu, void* stream);

/* Size of the fixed scratch of packmamba_causal_conv1d_bwd_noalloc, in bytes. */
#define PACKMAMBA_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

/*
 * packmamba_causal_conv1d_bwd without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid hipMalloc.  Same arguments (minus the workspace), results
 * and errors as packmamba_causal_conv1d_bwd, whose kernels it runs; the per-row
 * parameter-gradient partials live in a file-scope device array of
 * PACKMAMBA_NOALLOC_SCRATCH_BYTES that each GPU the library runs on holds until the
 * process ends.  The call itself allocates nothing (no hipMalloc, hipFree or
 * allocating library routine); the array's device address is looked up once per
 * device, on that device's first call.
 *   A shape whose packmamba_causal_conv1d_bwd_workspace_size() exceeds
 *   PACKMAMBA_NOALLOC_SCRATCH_BYTES returns PACKMAMBA_ERR_SCRATCH before anything
 *   is enqueued (e.g. batch * dim * (width + 1) * 4 bytes above 16 MiB for rows
 *   that are not split).
 *   Every call on a GPU shares that GPU's scratch and leaves its contents behind:
 *   calls that overlap on one GPU (concurrent streams, or threads) race and must
 *   be serialised by the caller.  Every scratch element a call reads is written
 *   by the same call first, so nothing needs clearing between calls.
 */
int packmamba_causal_conv1d_bwd_noalloc(const void* x, const float* weight, const float* bias,
                                        const int32_t* position_indices, const void* initial_x,
                                        const void* dout, const void* dfinal_x,
                                        void* dx, float* dweight, float* dbias, void* dinitial_x,
                                        int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
                                        int32_t dtype, int32_t silu, void* stream);

/* Bytes of the optional saved-states buffer of packmamba_selective_scan_fwd: the
 * chunk states, (batch, dim, ceil(seqlen / PACKMAMBA_STATE_STRIDE), dstate) floats,
 * then (batch, dim, seqlen rounded up to a multiple of 256) floats for the
 * backward's dz, in an order of the library's own, starting at the first multiple
 * of 256 bytes after the chunk states. */
size_t packmamba_selective_scan_fwd_saved_states_size(int64_t batch, int64_t dim, int64_t seqlen,
                                                      int32_t dstate);

/* Bytes of workspace packmamba_selective_scan_fwd needs: nonzero only for shapes
 * whose rows are split into segments scanned by separate blocks (long rows with
 * few batch rows and channels: fewer than 768 blocks of 16 channels); 0 when none
 * is needed or the shape is invalid (the call itself reports the latter). */
size_t packmamba_selective_scan_fwd_workspace_size(int64_t batch, int64_t dim, int64_t seqlen,
                                                   int32_t dstate);

/*
 * Packed selective scan, forward (Eqs. 1a, 1b, 2a; Alg. 2; §3.4).
 *   dt[b,d,l]   = softplus(delta[b,d,l] + delta_bias[d])   (softplus if delta_softplus,
 *                 identity above 20; delta_bias NULL means 0)
 *   Abar        = pos[b,l] == 0 ? 0 : exp(dt * A[d,n])      (reset at every sequence start)
 *   h[n]        = Abar * h[n] + dt * B[b,n,l] * u[b,d,l]     (h = 0 at every row start)
 *   y           = sum_n C[b,n,l] * h[n] + D[d] * u[b,d,l]   (D NULL means 0)
 *   out[b,d,l]  = z ? y * z * sigmoid(z) : y                 (z NULL means no gate)
 *   u, delta, z, out: dtype (batch, dim, seqlen); B, C: dtype (batch, dstate, seqlen);
 *   A (dim, dstate), D (dim), delta_bias (dim): float.  dstate must be 16.
 *   saved_states: NULL, or a float buffer of
 *   packmamba_selective_scan_fwd_saved_states_size() bytes that receives h after
 *   token min((c+1)*PACKMAMBA_STATE_STRIDE, seqlen)-1 for every chunk c, laid out
 *   (batch, dim, chunk, dstate), and, when z is given, (y + D u) times the
 *   derivative of z sigmoid(z) for every token after it: the factor of dout in dz.
 *   The backward reuses both instead of recomputing them.
 *   `out` may be NULL when saved_states or final_state is not (states only).
 *   initial_state: NULL (zeros), or (batch, dim, dstate) float: h before each row.
 *   final_state: NULL, or (batch, dim, dstate) float, receives h after each row.
 *   workspace: device scratch of packmamba_selective_scan_fwd_workspace_size()
 *   bytes, owned by the caller and not read after the call's kernels finish; may
 *   be NULL when that size is 0.  Too small or missing: PACKMAMBA_ERR_WORKSPACE.
 */
int packmamba_selective_scan_fwd(const void* u, const void* delta, const float* A,
                                 const void* B, const void* C, const float* D, const void* z,
                                 const float* delta_bias, int32_t delta_softplus,
                                 const int32_t* position_indices, const float* initial_state,
                                 void* out, float* final_state, float* saved_states,
                                 void* workspace, size_t workspace_bytes,
                                 int64_t batch, int64_t dim, int64_t seqlen, int32_t dstate,
                                 int32_t dtype, void* stream);

/* Bytes of workspace packmamba_selective_scan_bwd needs (includes room to
 * recompute the saved states when the caller passes none). */
size_t packmamba_selective_scan_bwd_workspace_size(int64_t batch, int64_t dim, int64_t seqlen,
                                                   int32_t dstate);

/*
 * Packed selective scan, backward (§3.4): gradients of sum(dout * out) for the
 * forward above.  The reverse recurrence
 *   dh_l = Abar_{l+1} * dh_{l+1} + C_l * dy_l,   Abar_{l+1} = 0 where token l+1 starts a sequence,
 * carries the matching reset; a reset multiplier is the constant 0, so no
 * gradient flows to delta or A through it.
 *   Inputs: as the forward, same order (initial_state included), plus dout
 *   (dtype), dfinal_state (NULL: zero; else the gradient of final_state,
 *   (batch, dim, dstate) float, entering h after the row's last token) and
 *   saved_states (NULL: recomputed into the workspace; else as written by the forward
 *   on the same inputs).
 *   Outputs (overwritten): du, ddelta (dtype, like u); dA (dim, dstate);
 *   dB, dC (batch, dstate, seqlen) float; dD (dim) iff D != NULL;
 *   dz (dtype) iff z != NULL; ddelta_bias (dim) iff delta_bias != NULL;
 *   dinitial_state (batch, dim, dstate) float iff initial_state != NULL.
 *   Sums over channels and tokens use per-block partials in the workspace and a
 *   second pass in fixed order: results are bitwise reproducible.
 */
int packmamba_selective_scan_bwd(const void* u, const void* delta, const float* A,
                                 const void* B, const void* C, const float* D, const void* z,
                                 const float* delta_bias, int32_t delta_softplus,
                                 const int32_t* position_indices, const float* initial_state,
                                 const void* dout, const float* dfinal_state,
                                 const float* saved_states,
                                 void* du, void* ddelta, float* dA, float* dB, float* dC,
                                 float* dD, void* dz, float* ddelta_bias, float* dinitial_state,
                                 void* workspace, size_t workspace_bytes,
                                 int64_t batch, int64_t dim, int64_t seqlen, int32_t dstate,
                                 int32_t dtype, void* stream);

/*
 * RMSNorm of the packed Mamba block (§3.2: a token-wise operator, which packing
 * leaves unchanged; no position indices are involved).  Over the feature axis of
 * x (batch, dim, seqlen), at every token:
 *   rstd[b,l] = 1 / sqrt(mean_d x[b,d,l]^2 + eps),  out = x * rstd * weight[d].
 *   weight (dim) float; rstd (batch, seqlen) float, written for the backward;
 *   out has x's shape and the dtype's output type.  eps >= 0 (PACKMAMBA_ERR_SHAPE
 *   otherwise).  Per-token sums use a fixed order.
 */
int packmamba_rmsnorm_fwd(const void* x, const float* weight, float eps, void* out, float* rstd,
                          int64_t batch, int64_t dim, int64_t seqlen, int32_t dtype, void* stream);

/* Bytes of workspace packmamba_rmsnorm_bwd needs. */
size_t packmamba_rmsnorm_bwd_workspace_size(int64_t batch, int64_t dim, int64_t seqlen);

/*
 * RMSNorm backward: with g = dout and s = sum_d g * weight * x at each token,
 *   dx = rstd * (g * weight - x * rstd^2 * s / dim) + dresidual,
 *   dweight[d] = sum_{b,l} g * x * rstd.
 *   x, dout, dresidual (NULL: none; the gradient reaching x through a residual
 *   connection) in the input type; dx in the output type; rstd as written by the
 *   forward; dweight (dim) float, overwritten.  The sum for dweight uses per-tile
 *   partials in the workspace and a second pass in fixed order (reproducible).
 */
int packmamba_rmsnorm_bwd(const void* x, const float* weight, const float* rstd, const void* dout,
                          const void* dresidual, void* dx, float* dweight, void* workspace,
                          size_t workspace_bytes, int64_t batch, int64_t dim, int64_t seqlen,
                          int32_t dtype, void* stream);

/*
 * Checks the index contract of §3.1 on the device: stores 1 to *d_flag (a device
 * int32 the caller zeroes beforehand) if any token violates
 * "pos[b,0] == 0 and pos[b,l] in {0, pos[b,l-1]+1}"; leaves it untouched otherwise.
 * With continued != 0, rows may continue a sequence: pos[b,0] >= 0 is accepted.
 */
int packmamba_check_position_indices(const int32_t* position_indices, int64_t batch,
                                     int64_t seqlen, int32_t continued, int32_t* d_flag,
                                     void* stream);

/*
 * Host-side packing plans (§3.1, §5).  Plain CPU functions on host memory: they
 * enqueue nothing and need no GPU.
 *
 * A plan places each sequence of a stream (lengths[i] tokens, in received order)
 * into rows of `seqlen` tokens as one or more pieces.  Policies:
 *   PACKMAMBA_PACK_SEQUENTIAL  in order; a sequence that does not fit the rest of
 *       the current row seals it, the rest being padding (§3.1, §5).  Sequences
 *       longer than a row are truncated to a row.
 *   PACKMAMBA_PACK_GREEDY      local greedy with a partial sort (§5): windows of
 *       `window` sequences, each sorted longest first and placed first-fit into
 *       the rows opened for that window, which are sealed when it ends.
 *       Truncates like the sequential policy.
 *   PACKMAMBA_PACK_CUT         the future work of §5: rows are filled to the end, a
 *       sequence that does not fit is cut at the row end and continues in the next
 *       row (first_pos > 0), so only the last row holds padding.  The operators'
 *       state passing makes this exact.
 * pieces: NULL to query the sizes (n_pieces, n_rows), else room for max_pieces
 * (PACKMAMBA_ERR_WORKSPACE if too few).  Errors: ERR_NULL, ERR_SHAPE (a length
 * <= 0, seqlen <= 0, window <= 0 for the greedy policy), ERR_UNSUPPORTED (policy).
 */
#define PACKMAMBA_PACK_SEQUENTIAL 0
#define PACKMAMBA_PACK_GREEDY 1
#define PACKMAMBA_PACK_CUT 2

typedef struct {
    int64_t seq;        /* index of the sequence in the stream */
    int64_t row;        /* row it is placed in */
    int64_t offset;     /* first token of the piece inside the row */
    int64_t length;     /* tokens in the piece */
    int64_t first_pos;  /* position of the piece's first token inside its sequence */
} packmamba_piece;

int packmamba_pack_plan(const int64_t* lengths, int64_t count, int64_t seqlen, int32_t policy,
                        int64_t window, packmamba_piece* pieces, int64_t max_pieces,
                        int64_t* n_pieces, int64_t* n_rows);

/*
 * Position indices (§3.1) of a plan, written to a host int32 array
 * (n_rows, seqlen): each piece gets first_pos, first_pos+1, ...; padding tokens get
 * index 0 (each its own sequence, so they affect nothing).  Rows that begin with a
 * piece whose first_pos > 0 continue a sequence (see state passing above).
 */
int packmamba_pack_positions(const packmamba_piece* pieces, int64_t n_pieces, int64_t n_rows,
                             int64_t seqlen, int32_t* position_indices);

#ifdef __cplusplus
}
#endif
#endif /* PACKMAMBA_H */
