/*
 * CPU reference ("oracle") for the Mixture of Channel Experts forward pass.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the HIP library; the HIP library never calls
 * it.
 *
 * Everything is plain loops in double precision over host memory.  Layout
 * codes: 0 = NCHW (x[b][c][p]), 1 = channels-last (x[b][p][c]), where p runs
 * over the H*W spatial positions (or the N tokens).  Element codes: 0 = float32,
 * 1 = bfloat16 bit patterns (uint16).
 */
#ifndef MOCE_ORACLE_H
#define MOCE_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Support preparation (Sec. 3.2 Eq. 2 fixed at inference; Sec. 3.3 input
 * order; Sec. 3.4 uncovered set U).  Returns -1 when every row is valid, the
 * index of the first invalid routed expert otherwise, or -2 for an invalid
 * shape (E < 1, E > C, k < 1, k > C).  On success s_out/w_out hold each row in
 * canonical order (logit descending, equal logits by ascending channel),
 * covered[c] is 1 for channels in some support, U lists the uncovered channels
 * ascending and *nU their count. */
int moce_oracle_prepare(int C, int E, int k, const int32_t* s, const float* w,
                        int32_t* s_out, float* w_out, uint8_t* covered,
                        int32_t* U, int32_t* nU);

/* Global average pooling descriptor (Sec. 3.3): d[b*C + c]. */
void moce_oracle_pool(int B, int C, int HW, int layout, int elem,
                      const void* x, double* d);

/* Temperature with the per-expert softplus-linear gate:
 * tau[b][o] = softplus(c[o] + sum_i a[o][i] * d[b][s[o][i]]) + 1e-3,
 * s in canonical order. */
void moce_oracle_gate_softplus(int B, int C, int E, int k, const double* d,
                               const int32_t* s, const float* a, const float* c,
                               double* tau);

/* Temperature with the paper's shared two-layer gate (Sec. 3.3 Eq. 3):
 * h = ReLU(W1 z_S + b1), g = w2 . h + b2,
 * tau = tau_min + (tau_max - tau_min) * sigmoid(g).  W1 is [k][k] row-major
 * (hidden unit j reads row j). */
void moce_oracle_gate_mlp(int B, int C, int E, int k, const double* d,
                          const int32_t* s, const float* W1, const float* b1,
                          const float* w2, float b2, float tau_min, float tau_max,
                          double* tau);

/* Mixing coefficients (Sec. 3.3 Eq. 4): alpha[b][o][i]. */
void moce_oracle_softmax(int B, int E, int k, const float* w, const double* tau,
                         double* alpha);

/* Routed outputs (Sec. 3.3 Eq. 5) and residual output (Sec. 3.4 Eq. 6).
 * y and mag use the layout of x with E output channels; the residual is
 * output channel E-1.  mag[..] = sum_i alpha_i |x_i| (routed) or the mean of
 * |x| over U (residual): the scale against which rounding error is judged. */
void moce_oracle_mix(int B, int C, int E, int k, int HW, int layout, int elem,
                     const void* x, const int32_t* s, const double* alpha,
                     const int32_t* U, int nU, double* y, double* mag);

/* Number of threads the OpenMP loops above use, and a setter (n >= 1). */
int moce_oracle_threads(void);
void moce_oracle_set_threads(int n);


/* Input-conditioned support (Sec. 4.5, Eq. 11).  The router's bottleneck
 * h[B][dd] = ReLU(Wh d + bh) from the descriptor d[B][C]; the example's
 * routing logits Lx[B][R][C] = L[R][C] + ((q[e] * h[b]) . v[c]); per row the k
 * largest logits in canonical order (ties to the lower channel) as channels
 * S[rows][k] and logits W[rows][k]; per example the uncovered channels
 * U[B][C] (first nU[b] entries, ascending). */
void moce_oracle_router(int B, int C, int dd, const double* d, const float* Wh,
                        const float* bh, double* h);
void moce_oracle_dynamic_logits(int B, int C, int R, int dd, const double* h, const float* L,
                                const float* q, const float* v, double* Lx);
void moce_oracle_topk(int rows, int C, int k, const double* Lx, int32_t* S, double* W);
void moce_oracle_dynamic_uncovered(int B, int C, int R, int k, const int32_t* S, int32_t* U, int32_t* nU);

#ifdef __cplusplus
}
#endif

#endif
