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
 * Optional inputs (bias, D, z, delta_bias) may be NULL; their gradient pointers
 * are then ignored.  Gradient outputs are fully overwritten (not accumulated).
 */
#ifndef PACKMAMBA_ORACLE_H
#define PACKMAMBA_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Alg. 1 (conv1d_pack), forward: causal depthwise conv whose taps stop at the
 * start of the output token's own sequence, plus bias, optionally SiLU. */
void pmo_conv1d_fwd(const double* x, const double* w, const double* bias,
                    const int32_t* pos, double* out,
                    int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
                    int32_t silu);

/* §3.3, conv1d_pack backward: dx (the exact adjoint of the masked forward), dw, dbias. */
void pmo_conv1d_bwd(const double* x, const double* w, const double* bias,
                    const int32_t* pos, const double* dout,
                    double* dx, double* dw, double* dbias,
                    int64_t batch, int64_t dim, int64_t seqlen, int32_t width,
                    int32_t silu);

/* Eqs. (1a), (1b), (2a) with the reset of Alg. 2 / §3.4 (the multiplier is 0 at
 * position index 0), plus the D skip, the SiLU(z) gate and softplus on delta. */
void pmo_scan_fwd(const double* u, const double* delta, const double* A,
                  const double* B, const double* C, const double* D,
                  const double* z, const double* delta_bias, int32_t delta_softplus,
                  const int32_t* pos, double* out,
                  int64_t batch, int64_t dim, int64_t seqlen, int32_t dstate);

/* Hidden state h after token min((c+1)*stride, seqlen)-1 for every chunk c:
 * states is (batch, dim, ceil(seqlen/stride), dstate). */
void pmo_scan_states(const double* u, const double* delta, const double* A,
                     const double* B, const double* delta_bias, int32_t delta_softplus,
                     const int32_t* pos, double* states,
                     int64_t batch, int64_t dim, int64_t seqlen, int32_t dstate,
                     int64_t stride);

/* §3.4 backward: gradients of sum(dout * out) with respect to every input. */
void pmo_scan_bwd(const double* u, const double* delta, const double* A,
                  const double* B, const double* C, const double* D,
                  const double* z, const double* delta_bias, int32_t delta_softplus,
                  const int32_t* pos, const double* dout,
                  double* du, double* ddelta, double* dA, double* dB, double* dC,
                  double* dD, double* dz, double* ddelta_bias,
                  int64_t batch, int64_t dim, int64_t seqlen, int32_t dstate);

/* Index contract of §3.1: every row starts a sequence and each index is 0 or the
 * previous index plus one.  Returns -1 if valid, else the flat index of the first
 * violation. */
int64_t pmo_check_positions(const int32_t* pos, int64_t batch, int64_t seqlen);

/* Number of OpenMP threads the oracle runs with (1 without OpenMP). */
int32_t pmo_num_threads(void);

/* Set the number of OpenMP threads (no effect without OpenMP). */
void pmo_set_num_threads(int32_t n);

#ifdef __cplusplus
}
#endif
#endif
