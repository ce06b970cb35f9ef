/*
 * oracle.c -- fp64 CPU reference for PackMamba's sequence-wise operators.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker, not the product: only the
 * tests, the smoke check and the benchmark's CPU-baseline leg use it.  It is a
 * plain sequential recurrence per (batch row, channel), written from the paper's
 * definitions, with no blocking, fusion or reordering beyond them.  Rows are
 * independent, so OpenMP runs them in parallel; nothing else is parallel.
 *
 * Readings of the paper that this file takes (each also listed in the design notes):
 *  - Alg. 1 leaves the weight index undefined for indices >= width and loops one
 *    tap too far; the reading here is: the tap that reaches k tokens back is used
 *    iff k <= position index of the output token (and the tap stays in the row);
 *    weight[d, width-1] multiplies the current token.
 *  - B-bar x is the simplified product delta * B * x of Alg. 2 (not the ZOH form
 *    of Eq. 2b).  A is real, diagonal per channel: A-bar = exp(delta * A[d,n]).
 *  - The reset sets A-bar to the constant 0 where the position index is 0
 *    (Alg. 2, §3.4), so no gradient flows through a reset multiplier; every row
 *    also starts from h = 0.
 *  - The readout adds the D skip and gates with SiLU(z); delta gets delta_bias
 *    and softplus (threshold 20, above which softplus is the identity).
 *  - State passing across rows (the future work of §5: a sequence cut at a row
 *    end continues in another row): optional per-row initial and final states.
 *    For the conv they are the width-1 inputs before the row and the row's last
 *    width-1 inputs; for the scan, h before the row's first token and h after its
 *    last.  A row whose first position index is not 0 continues a sequence; a
 *    start (index 0) still cuts everything before it, the initial state included.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double sigmoid(double v) { return 1.0 / (1.0 + exp(-v)); }

/* softplus with the identity above the threshold 20 */
static double softplus(double s) { return s > 20.0 ? s : log1p(exp(s)); }
static double softplus_grad(double s) { return s > 20.0 ? 1.0 : sigmoid(s); }

int32_t pmo_num_threads(void) {
#ifdef _OPENMP
    return (int32_t)omp_get_max_threads();
#else
    return 1;
#endif
}

void pmo_set_num_threads(int32_t n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------------- */
/* causal conv1d with sequence-start masking (Alg. 1, §3.3)                  */
/* ------------------------------------------------------------------------- */

/* input of token m of one (b, d) row; m < 0 reads the row's initial inputs
 * xi (width-1 of them, token -1 last), or 0 without them */
static double x_at(const double* xr, const double* xi, int32_t width, int64_t m) {
    if (m >= 0) return xr[m];
    return xi ? xi[width - 1 + m] : 0.0;
}

/* pre-activation of output token l of one (b, d) row */
static double conv_pre(const double* xr, const double* xi, const double* wd, double b0,
                       const int32_t* pr, int64_t l, int32_t width) {
    double acc = b0;
    for (int32_t k = 0; k < width; ++k) {           /* tap reaching k tokens back */
        if (k > pr[l]) break;                       /* before the token's own sequence */
        acc += wd[width - 1 - k] * x_at(xr, xi, width, l - k);
    }
    return acc;
}

void pmo_conv1d_fwd(const double* x, const double* w, const double* bias,
                    const int32_t* pos, const double* xinit, double* out, double* xfinal,
                    int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
                    int32_t silu) {
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < batch; ++b) {
        for (int64_t d = 0; d < dim; ++d) {
            const double* xr = x + (b * dim + d) * seqlen;
            const double* xi = xinit ? xinit + (b * dim + d) * (width - 1) : NULL;
            const int32_t* pr = pos + b * seqlen;
            double* orow = out + (b * dim + d) * seqlen;
            const double b0 = bias ? bias[d] : 0.0;
            for (int64_t l = 0; l < seqlen; ++l) {
                const double v = conv_pre(xr, xi, w + d * width, b0, pr, l, width);
                orow[l] = silu ? v * sigmoid(v) : v;
            }
            /* the row's last width-1 inputs (reaching into xi when the row is shorter) */
            if (xfinal)
                for (int32_t i = 0; i < width - 1; ++i)
                    xfinal[(b * dim + d) * (width - 1) + i] = x_at(xr, xi, width, seqlen - (width - 1) + i);
        }
    }
}

void pmo_conv1d_bwd(const double* x, const double* w, const double* bias,
                    const int32_t* pos, const double* xinit, const double* dout,
                    const double* dxfinal, double* dx, double* dw, double* dbias,
                    double* dxinit,
                    int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
                    int32_t silu) {
#pragma omp parallel for schedule(static)
    for (int64_t d = 0; d < dim; ++d) {
        const double* wd = w + d * width;
        double* dwd = dw + d * width;
        double db = 0.0;
        for (int32_t j = 0; j < width; ++j) dwd[j] = 0.0;
        for (int64_t b = 0; b < batch; ++b) {
            const double* xr = x + (b * dim + d) * seqlen;
            const double* gr = dout + (b * dim + d) * seqlen;
            const int32_t* pr = pos + b * seqlen;
            const double* xi = xinit ? xinit + (b * dim + d) * (width - 1) : NULL;
            double* dxr = dx + (b * dim + d) * seqlen;
            double* dxi = (xinit && dxinit) ? dxinit + (b * dim + d) * (width - 1) : NULL;
            const double b0 = bias ? bias[d] : 0.0;
            for (int64_t l = 0; l < seqlen; ++l) dxr[l] = 0.0;
            if (dxi)
                for (int32_t i = 0; i < width - 1; ++i) dxi[i] = 0.0;
            for (int64_t l = 0; l < seqlen; ++l) {
                double g = gr[l];
                if (silu) {
                    const double v = conv_pre(xr, xi, wd, b0, pr, l, width);
                    const double s = sigmoid(v);
                    g *= s * (1.0 + v * (1.0 - s));
                }
                db += g;
                /* adjoint of the forward taps: the same mask, scattered back */
                for (int32_t k = 0; k < width; ++k) {
                    if (k > pr[l]) break;
                    if (l - k >= 0) {
                        dxr[l - k] += wd[width - 1 - k] * g;
                    } else if (dxi) {
                        dxi[width - 1 + l - k] += wd[width - 1 - k] * g;
                    }
                    dwd[width - 1 - k] += g * x_at(xr, xi, width, l - k);
                }
            }
            /* the final inputs are copies of the last width-1 inputs */
            if (dxfinal)
                for (int32_t i = 0; i < width - 1; ++i) {
                    const int64_t m = seqlen - (width - 1) + i;
                    const double gf = dxfinal[(b * dim + d) * (width - 1) + i];
                    if (m >= 0) dxr[m] += gf;
                    else if (dxi) dxi[width - 1 + m] += gf;
                }
        }
        if (dbias) dbias[d] = db;
    }
}

/* ------------------------------------------------------------------------- */
/* selective scan with resets (Eqs. 1a, 1b, 2a; Alg. 2; §3.4)                 */
/* ------------------------------------------------------------------------- */

static double step_size(const double* delta_row, const double* delta_bias, int32_t sp,
                        int64_t d, int64_t l) {
    const double s = delta_row[l] + (delta_bias ? delta_bias[d] : 0.0);
    return sp ? softplus(s) : s;
}

/* one (b, d) row forward from the state h0 (NULL: 0); writes h for every token into
 * hs (seqlen x dstate) and the multipliers into as_ when they are non-NULL */
static void scan_row_forward(const double* ur, const double* dr, const double* Ad,
                             const double* Bb, const int32_t* pr,
                             const double* delta_bias, int32_t sp, int64_t d,
                             int64_t seqlen, int32_t N, const double* h0, double* h,
                             double* hs, double* as_, double* dts) {
    for (int32_t n = 0; n < N; ++n) h[n] = h0 ? h0[n] : 0.0;
    for (int64_t l = 0; l < seqlen; ++l) {
        const double dt = step_size(dr, delta_bias, sp, d, l);
        if (dts) dts[l] = dt;
        for (int32_t n = 0; n < N; ++n) {
            const double a = (pr[l] == 0) ? 0.0 : exp(dt * Ad[n]);   /* reset: A-bar -> 0 */
            h[n] = a * h[n] + dt * Bb[(int64_t)n * seqlen + l] * ur[l];
            if (as_) as_[l * N + n] = a;
            if (hs) hs[l * N + n] = h[n];
        }
    }
}

void pmo_scan_fwd(const double* u, const double* delta, const double* A,
                  const double* B, const double* C, const double* D,
                  const double* z, const double* delta_bias, int32_t delta_softplus,
                  const int32_t* pos, const double* h0, double* out, double* hfinal,
                  int64_t batch, int64_t dim, int64_t seqlen, int32_t dstate) {
    const int32_t N = dstate;
#pragma omp parallel
    {
        double* h = (double*)malloc(sizeof(double) * N);
#pragma omp for collapse(2) schedule(static)
        for (int64_t b = 0; b < batch; ++b) {
            for (int64_t d = 0; d < dim; ++d) {
                const int64_t row = (b * dim + d) * seqlen;
                const double* ur = u + row;
                const double* dr = delta + row;
                const double* Bb = B + b * N * seqlen;
                const double* Cb = C + b * N * seqlen;
                const int32_t* pr = pos + b * seqlen;
                for (int32_t n = 0; n < N; ++n) h[n] = h0 ? h0[(b * dim + d) * N + n] : 0.0;
                for (int64_t l = 0; l < seqlen; ++l) {
                    const double dt = step_size(dr, delta_bias, delta_softplus, d, l);
                    double y = 0.0;
                    for (int32_t n = 0; n < N; ++n) {
                        const double a = (pr[l] == 0) ? 0.0 : exp(dt * A[d * N + n]);
                        h[n] = a * h[n] + dt * Bb[(int64_t)n * seqlen + l] * ur[l];
                        y += Cb[(int64_t)n * seqlen + l] * h[n];
                    }
                    const double yD = y + (D ? D[d] * ur[l] : 0.0);
                    out[row + l] = z ? yD * z[row + l] * sigmoid(z[row + l]) : yD;
                }
                if (hfinal)
                    for (int32_t n = 0; n < N; ++n) hfinal[(b * dim + d) * N + n] = h[n];
            }
        }
        free(h);
    }
}

void pmo_scan_states(const double* u, const double* delta, const double* A,
                     const double* B, const double* delta_bias, int32_t delta_softplus,
                     const int32_t* pos, const double* h0, double* states,
                     int64_t batch, int64_t dim, int64_t seqlen, int32_t dstate,
                     int64_t stride) {
    const int32_t N = dstate;
    const int64_t nchunk = (seqlen + stride - 1) / stride;
#pragma omp parallel
    {
        double* h = (double*)malloc(sizeof(double) * N);
        double* hs = (double*)malloc(sizeof(double) * N * seqlen);
#pragma omp for collapse(2) schedule(static)
        for (int64_t b = 0; b < batch; ++b) {
            for (int64_t d = 0; d < dim; ++d) {
                const int64_t row = (b * dim + d) * seqlen;
                scan_row_forward(u + row, delta + row, A + d * N, B + b * N * seqlen,
                                 pos + b * seqlen, delta_bias, delta_softplus, d, seqlen, N,
                                 h0 ? h0 + (b * dim + d) * N : NULL, h, hs, NULL, NULL);
                for (int64_t c = 0; c < nchunk; ++c) {
                    int64_t last = (c + 1) * stride;
                    if (last > seqlen) last = seqlen;
                    for (int32_t n = 0; n < N; ++n)
                        states[((b * dim + d) * nchunk + c) * N + n] = hs[(last - 1) * N + n];
                }
            }
        }
        free(hs);
        free(h);
    }
}

void pmo_scan_bwd(const double* u, const double* delta, const double* A,
                  const double* B, const double* C, const double* D,
                  const double* z, const double* delta_bias, int32_t delta_softplus,
                  const int32_t* pos, const double* h0, const double* dout,
                  const double* dhfinal,
                  double* du, double* ddelta, double* dA, double* dB, double* dC,
                  double* dD, double* dz, double* ddelta_bias, double* dh0,
                  int64_t batch, int64_t dim, int64_t seqlen, int32_t dstate) {
    const int32_t N = dstate;
    const int64_t bc = batch * N * seqlen;          /* size of dB (and dC) */
    const int nth = pmo_num_threads();
    /* dB and dC sum over channels; each thread accumulates privately, then the
     * private buffers are added in thread order */
    double* priv = (double*)calloc((size_t)nth * 2 * (size_t)bc, sizeof(double));

#pragma omp parallel
    {
        int tid = 0;
#ifdef _OPENMP
        tid = omp_get_thread_num();
#endif
        double* dBt = priv + (size_t)tid * 2 * bc;
        double* dCt = dBt + bc;
        double* h = (double*)malloc(sizeof(double) * N);
        double* hs = (double*)malloc(sizeof(double) * N * seqlen);
        double* as_ = (double*)malloc(sizeof(double) * N * seqlen);
        double* dts = (double*)malloc(sizeof(double) * seqlen);
        double* dy = (double*)malloc(sizeof(double) * seqlen);
        double* ddt = (double*)malloc(sizeof(double) * seqlen);
        double* dh = (double*)malloc(sizeof(double) * N);

#pragma omp for schedule(static)
        for (int64_t d = 0; d < dim; ++d) {
            double dDd = 0.0, ddbd = 0.0;
            for (int32_t n = 0; n < N; ++n) dA[d * N + n] = 0.0;
            for (int64_t b = 0; b < batch; ++b) {
                const int64_t row = (b * dim + d) * seqlen;
                const double* ur = u + row;
                const double* dr = delta + row;
                const double* Bb = B + b * N * seqlen;
                const double* Cb = C + b * N * seqlen;
                const int32_t* pr = pos + b * seqlen;
                double* dBb = dBt + b * N * seqlen;
                double* dCb = dCt + b * N * seqlen;

                const double* h0r = h0 ? h0 + (b * dim + d) * N : NULL;
                scan_row_forward(ur, dr, A + d * N, Bb, pr, delta_bias, delta_softplus,
                                 d, seqlen, N, h0r, h, hs, as_, dts);

                /* gate and skip: out = yD * SiLU(z), yD = y + D u, y = sum_n C h */
                for (int64_t l = 0; l < seqlen; ++l) {
                    double y = 0.0;
                    for (int32_t n = 0; n < N; ++n) y += Cb[(int64_t)n * seqlen + l] * hs[l * N + n];
                    const double yD = y + (D ? D[d] * ur[l] : 0.0);
                    const double g = dout[row + l];
                    double dyD = g;
                    if (z) {
                        const double zz = z[row + l], s = sigmoid(zz);
                        dz[row + l] = g * yD * s * (1.0 + zz * (1.0 - s));
                        dyD = g * zz * s;
                    }
                    dy[l] = dyD;
                    du[row + l] = D ? dyD * D[d] : 0.0;
                    if (D) dDd += dyD * ur[l];
                    for (int32_t n = 0; n < N; ++n) dCb[(int64_t)n * seqlen + l] += dyD * hs[l * N + n];
                    ddt[l] = 0.0;
                }

                /* reverse recurrence dh_l = A-bar_{l+1} dh_{l+1} + C_l dy_l, where
                 * A-bar_{l+1} is 0 when token l+1 starts a sequence (as stored); past
                 * the row end, "dh" is the final state's gradient, which h_{L-1}
                 * receives with multiplier 1 */
                for (int32_t n = 0; n < N; ++n) dh[n] = dhfinal ? dhfinal[(b * dim + d) * N + n] : 0.0;
                for (int64_t l = seqlen - 1; l >= 0; --l) {
                    const double dt = dts[l];
                    for (int32_t n = 0; n < N; ++n) {
                        const double an = (l + 1 < seqlen) ? as_[(l + 1) * N + n] : 1.0;
                        const double Bl = Bb[(int64_t)n * seqlen + l];
                        dh[n] = dy[l] * Cb[(int64_t)n * seqlen + l] + an * dh[n];
                        dBb[(int64_t)n * seqlen + l] += dh[n] * dt * ur[l];
                        du[row + l] += dh[n] * dt * Bl;
                        ddt[l] += dh[n] * Bl * ur[l];
                        if (pr[l] != 0) {
                            /* A-bar_l = exp(dt_l A[d,n]) depends on dt_l and A; the state
                             * before the row's first token is h0 (or 0) */
                            const double hp = l > 0 ? hs[(l - 1) * N + n] : (h0r ? h0r[n] : 0.0);
                            const double t = dh[n] * hp * as_[l * N + n];
                            ddt[l] += t * A[d * N + n];
                            dA[d * N + n] += t * dt;
                        }
                    }
                    double gs = 1.0;
                    if (delta_softplus)
                        gs = softplus_grad(dr[l] + (delta_bias ? delta_bias[d] : 0.0));
                    ddelta[row + l] = ddt[l] * gs;
                    ddbd += ddelta[row + l];
                }
                /* dh now holds dh_0; h0 reaches h_0 through A-bar_0 (0 at a start) */
                if (h0r && dh0)
                    for (int32_t n = 0; n < N; ++n) dh0[(b * dim + d) * N + n] = as_[n] * dh[n];
            }
            if (D && dD) dD[d] = dDd;
            if (delta_bias && ddelta_bias) ddelta_bias[d] = ddbd;
        }
        free(dh); free(ddt); free(dy); free(dts); free(as_); free(hs); free(h);
    }

    for (int64_t i = 0; i < bc; ++i) { dB[i] = 0.0; dC[i] = 0.0; }
    for (int t = 0; t < nth; ++t) {
        const double* dBt = priv + (size_t)t * 2 * bc;
        const double* dCt = dBt + bc;
        for (int64_t i = 0; i < bc; ++i) { dB[i] += dBt[i]; dC[i] += dCt[i]; }
    }
    free(priv);
}

int64_t pmo_check_positions(const int32_t* pos, int64_t batch, int64_t seqlen,
                            int32_t continued) {
    for (int64_t b = 0; b < batch; ++b) {
        const int32_t* pr = pos + b * seqlen;
        for (int64_t l = 0; l < seqlen; ++l) {
            const int ok = (l == 0) ? (continued ? pr[l] >= 0 : pr[l] == 0)
                                    : (pr[l] == 0 || pr[l] == pr[l - 1] + 1);
            if (!ok) return b * seqlen + l;
        }
    }
    return -1;
}
