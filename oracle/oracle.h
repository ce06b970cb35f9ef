/*
 * oracle.h -- fp64 CPU reference for PackMamba's two sequence-wise operators.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg may call this library; the HIP path never links or calls it,
 * and it shares no code, header or table with that path.
 *
 * Every array is contiguous row-major fp64 (int32 for position indices) with the
 * sequence axis innermost:
 *   activations x, u, delta, z, dout, outputs   (batch, dim, seqlen)
 *   B, C and their gradients                    (batch, dstate, seqlen)
 *   A and dA                                    (dim, dstate)
 *   conv weight w and dw                        (dim, width)
 *   D, delta_bias, conv bias and gradients      (dim)
 *   position_indices                            (batch, seqlen)
 *   conv initial/final inputs and gradients     (batch, dim, width-1), token -1 last
 *   scan initial/final states and gradients     (batch, dim, dstate)
 * Optional inputs (bias, D, z, delta_bias, the initial states) may be NULL; their
 * gradient pointers are then ignored.  A NULL final-state gradient means 0.
 * Gradient outputs are fully overwritten (not accumulated).
 *
 * State passing across rows (§5, future work): a row may continue a sequence cut
 * at the end of another row.  Its first position index is then that token's
 * position inside the sequence, and the initial states carry the other part's
 * final states in; without them the continued sequence sees zeros.
 */
#ifndef PACKMAMBA_ORACLE_H
#define PACKMAMBA_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Alg. 1 (conv1d_pack), forward: causal depthwise conv whose taps stop at the
 * start of the output token's own sequence, plus bias, optionally SiLU.  Taps
 * reaching before the row read xinit (NULL: zeros); xfinal (may be NULL)
 * receives the row's last width-1 inputs. */
void pmo_conv1d_fwd(const double* x, const double* w, const double* bias,
                    const int32_t* pos, const double* xinit, double* out, double* xfinal,
                    int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
                    int32_t silu);

/* §3.3, conv1d_pack backward: dx (the exact adjoint of the masked forward), dw,
 * dbias, and dxinit when xinit is given; dxfinal is the gradient of xfinal. */
void pmo_conv1d_bwd(const double* x, const double* w, const double* bias,
                    const int32_t* pos, const double* xinit, const double* dout,
                    const double* dxfinal, double* dx, double* dw, double* dbias,
                    double* dxinit,
                    int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
                    int32_t silu);

/* Eqs. (1a), (1b), (2a) with the reset of Alg. 2 / §3.4 (the multiplier is 0 at
 * position index 0), plus the D skip, the SiLU(z) gate and softplus on delta.
 * h starts from h0 (NULL: 0); hfinal (may be NULL) receives h after the last token. */
void pmo_scan_fwd(const double* u, const double* delta, const double* A,
                  const double* B, const double* C, const double* D,
                  const double* z, const double* delta_bias, int32_t delta_softplus,
                  const int32_t* pos, const double* h0, double* out, double* hfinal,
                  int64_t batch, int64_t dim, int64_t seqlen, int32_t dstate);

/* Hidden state h after token min((c+1)*stride, seqlen)-1 for every chunk c:
 * states is (batch, dim, ceil(seqlen/stride), dstate). */
void pmo_scan_states(const double* u, const double* delta, const double* A,
                     const double* B, const double* delta_bias, int32_t delta_softplus,
                     const int32_t* pos, const double* h0, double* states,
                     int64_t batch, int64_t dim, int64_t seqlen, int32_t dstate,
                     int64_t stride);

/* §3.4 backward: gradients of sum(dout * out) + sum(dhfinal * hfinal) with respect
 * to every input, dh0 included when h0 is given. */
void pmo_scan_bwd(const double* u, const double* delta, const double* A,
                  const double* B, const double* C, const double* D,
                  const double* z, const double* delta_bias, int32_t delta_softplus,
                  const int32_t* pos, const double* h0, const double* dout,
                  const double* dhfinal,
                  double* du, double* ddelta, double* dA, double* dB, double* dC,
                  double* dD, double* dz, double* ddelta_bias, double* dh0,
                  int64_t batch, int64_t dim, int64_t seqlen, int32_t dstate);

/* Index contract of §3.1: every row starts a sequence (with continued != 0: its
 * first index may be any value >= 0, a sequence carried over from another row)
 * and each later index is 0 or the previous index plus one.  Returns -1 if valid,
 * else the flat index of the first violation. */
int64_t pmo_check_positions(const int32_t* pos, int64_t batch, int64_t seqlen,
                            int32_t continued);

/* Number of OpenMP threads the oracle runs with (1 without OpenMP). */
int32_t pmo_num_threads(void);

/* Set the number of OpenMP threads (no effect without OpenMP). */
void pmo_set_num_threads(int32_t n);

#ifdef __cplusplus
}
#endif
#endif
