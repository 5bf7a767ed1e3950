/*
 * CPU reference ("oracle") for the Mixture of Channel Experts forward pass.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests, the smoke check and the
 * benchmark's CPU-baseline leg, never by the HIP library.
 *
 * Each function is the paper's definition written out as plain loops in
 * double precision.  The only parallelism is an OpenMP loop over images, which
 * does not change any result (every image is computed by one thread, in the
 * same order).
 *
 * Readings taken where the paper leaves a choice open:
 *  - the gate's k inputs are the support descriptors in descending routing
 *    logit order (Sec. 3.3); equal logits go to the lower channel first;
 *  - the softmax of Eq. 4 subtracts the largest scaled logit before
 *    exponentiating, which leaves every coefficient unchanged mathematically
 *    and keeps very small temperatures finite;
 *  - the residual output of Eq. 6 is the last output channel;
 *  - the softplus-linear temperature tau = softplus(a_o . z_S + c_o) + 1e-3 is
 *    provided beside the paper's shared two-layer gate (Eq. 3).
 */
#include "moce_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int moce_oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void moce_oracle_set_threads(int n) {
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Exact widening of one input element to double. */
static double load_x(const void* x, int elem, size_t idx) {
    if (elem == 0) return (double)((const float*)x)[idx];
    uint32_t bits = (uint32_t)((const uint16_t*)x)[idx] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static size_t x_index(int layout, int C, int HW, int b, int c, int p) {
    if (layout == 0) return ((size_t)b * C + c) * HW + p;
    return ((size_t)b * HW + p) * C + c;
}

/* ------------------------------------------------------------------------ */
/* Static support at inference (Sec. 3.2, Eq. 2) and uncovered set (Sec. 3.4) */

/* a precedes b in the canonical order: larger logit first, then lower channel */
static int comes_before(float wa, int32_t sa, float wb, int32_t sb) {
    if (wa > wb) return 1;
    if (wa < wb) return 0;
    return sa < sb;
}

int moce_oracle_prepare(int C, int E, int k, const int32_t* s, const float* w,
                        int32_t* s_out, float* w_out, uint8_t* covered,
                        int32_t* U, int32_t* nU) {
    if (E < 1 || E > C || k < 1 || k > C) return -2;
    const int R = E - 1;

    /* A support is TopK of one logit row: k distinct channels of [0, C) with
     * finite logits.  Report the first routed expert that violates this. */
    for (int o = 0; o < R; ++o) {
        for (int i = 0; i < k; ++i) {
            int32_t ch = s[(size_t)o * k + i];
            float lg = w[(size_t)o * k + i];
            if (ch < 0 || ch >= C || !isfinite(lg)) return o;
            for (int j = 0; j < i; ++j)
                if (s[(size_t)o * k + j] == ch) return o;
        }
    }

    /* Canonical order of each row, by insertion sort (stable). */
    for (int o = 0; o < R; ++o) {
        int32_t* so = s_out + (size_t)o * k;
        float* wo = w_out + (size_t)o * k;
        for (int i = 0; i < k; ++i) {
            int32_t ch = s[(size_t)o * k + i];
            float lg = w[(size_t)o * k + i];
            int j = i;
            while (j > 0 && comes_before(lg, ch, wo[j - 1], so[j - 1])) {
                so[j] = so[j - 1];
                wo[j] = wo[j - 1];
                --j;
            }
            so[j] = ch;
            wo[j] = lg;
        }
    }

    /* U = {0..C-1} minus the union of all supports, ascending. */
    memset(covered, 0, (size_t)C);
    for (size_t t = 0; t < (size_t)R * k; ++t) covered[s[t]] = 1;
    int n = 0;
    for (int c = 0; c < C; ++c)
        if (!covered[c]) U[n++] = c;
    *nU = n;
    return -1;
}

/* ------------------------------------------------------------------------ */
/* Global average pooling, z = GAP(X) (Sec. 3.3) */

void moce_oracle_pool(int B, int C, int HW, int layout, int elem,
                      const void* x, double* d) {
    #pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int c = 0; c < C; ++c) {
            double sum = 0.0;
            for (int p = 0; p < HW; ++p) sum += load_x(x, elem, x_index(layout, C, HW, b, c, p));
            d[(size_t)b * C + c] = sum / (double)HW;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Temperatures (Sec. 3.3) */

static double softplus(double t) {
    /* log(1 + e^t), written so that neither branch overflows */
    return fmax(t, 0.0) + log1p(exp(-fabs(t)));
}

void moce_oracle_gate_softplus(int B, int C, int E, int k, const double* d,
                               const int32_t* s, const float* a, const float* c,
                               double* tau) {
    const int R = E - 1;
    #pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int o = 0; o < R; ++o) {
            double g = (double)c[o];
            for (int i = 0; i < k; ++i)
                g += (double)a[(size_t)o * k + i] * d[(size_t)b * C + s[(size_t)o * k + i]];
            tau[(size_t)b * R + o] = softplus(g) + 1e-3;
        }
    }
}

void moce_oracle_gate_mlp(int B, int C, int E, int k, const double* d,
                          const int32_t* s, const float* W1, const float* b1,
                          const float* w2, float b2, float tau_min, float tau_max,
                          double* tau) {
    const int R = E - 1;
    #pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        double* z = (double*)malloc(sizeof(double) * (size_t)k);
        for (int o = 0; o < R; ++o) {
            /* gate input: the support's descriptors, position i = i-th preferred */
            for (int i = 0; i < k; ++i) z[i] = d[(size_t)b * C + s[(size_t)o * k + i]];
            double g = (double)b2;
            for (int j = 0; j < k; ++j) {
                double h = (double)b1[j];
                for (int i = 0; i < k; ++i) h += (double)W1[(size_t)j * k + i] * z[i];
                if (h < 0.0) h = 0.0;
                g += (double)w2[j] * h;
            }
            double sig = 1.0 / (1.0 + exp(-g));
            tau[(size_t)b * R + o] = (double)tau_min + ((double)tau_max - (double)tau_min) * sig;
        }
        free(z);
    }
}

/* ------------------------------------------------------------------------ */
/* Mixing coefficients, Eq. 4 */

void moce_oracle_softmax(int B, int E, int k, const float* w, const double* tau,
                         double* alpha) {
    const int R = E - 1;
    #pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int o = 0; o < R; ++o) {
            const double t = tau[(size_t)b * R + o];
            const float* wo = w + (size_t)o * k;
            double* al = alpha + ((size_t)b * R + o) * k;
            double m = -INFINITY;
            for (int i = 0; i < k; ++i)
                if ((double)wo[i] / t > m) m = (double)wo[i] / t;
            double z = 0.0;
            for (int i = 0; i < k; ++i) {
                al[i] = exp((double)wo[i] / t - m);
                z += al[i];
            }
            for (int i = 0; i < k; ++i) al[i] /= z;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Routed experts (Eq. 5) and residual aggregate (Eq. 6) */

void moce_oracle_mix(int B, int C, int E, int k, int HW, int layout, int elem,
                     const void* x, const int32_t* s, const double* alpha,
                     const int32_t* U, int nU, double* y, double* mag) {
    const int R = E - 1;
    #pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int o = 0; o < R; ++o) {
            const double* al = alpha + ((size_t)b * R + o) * k;
            const int32_t* so = s + (size_t)o * k;
            for (int p = 0; p < HW; ++p) {
                double acc = 0.0, m = 0.0;
                for (int i = 0; i < k; ++i) {
                    double v = load_x(x, elem, x_index(layout, C, HW, b, so[i], p));
                    acc += al[i] * v;
                    m += al[i] * fabs(v);
                }
                size_t yi = x_index(layout, E, HW, b, o, p);
                y[yi] = acc;
                mag[yi] = m;
            }
        }
        for (int p = 0; p < HW; ++p) {
            double acc = 0.0, m = 0.0;
            for (int j = 0; j < nU; ++j) {
                double v = load_x(x, elem, x_index(layout, C, HW, b, U[j], p));
                acc += v;
                m += fabs(v);
            }
            size_t yi = x_index(layout, E, HW, b, E - 1, p);
            y[yi] = nU > 0 ? acc / (double)nU : 0.0;
            mag[yi] = nU > 0 ? m / (double)nU : 0.0;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Input-conditioned (dynamic) support (Sec. 4.5, Eq. 11)                     */

/* h[b][t] = ReLU(bh[t] + sum_c Wh[t][c] d[b][c]), the router's bottleneck. */
void moce_oracle_router(int B, int C, int dd, const double* d, const float* Wh,
                        const float* bh, double* h) {
    #pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int t = 0; t < dd; ++t) {
            double acc = bh[t];
            for (int c = 0; c < C; ++c) acc += (double)Wh[(size_t)t * C + c] * d[(size_t)b * C + c];
            h[(size_t)b * dd + t] = acc > 0.0 ? acc : 0.0;
        }
    }
}

/* Lx[b][e][c] = L[e][c] + sum_t q[e][t] h[b][t] v[c][t]: the static routing
 * logits plus the rank-dd offset of example b. */
void moce_oracle_dynamic_logits(int B, int C, int R, int dd, const double* h, const float* L,
                                const float* q, const float* v, double* Lx) {
    #pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int e = 0; e < R; ++e) {
            for (int c = 0; c < C; ++c) {
                double off = 0.0;
                for (int t = 0; t < dd; ++t)
                    off += (double)q[(size_t)e * dd + t] * h[(size_t)b * dd + t] * (double)v[(size_t)c * dd + t];
                Lx[((size_t)b * R + e) * C + c] = (double)L[(size_t)e * C + c] + off;
            }
        }
    }
}

/* a precedes b: larger logit first, then lower channel */
static int comes_before_d(double wa, int32_t sa, double wb, int32_t sb) {
    if (wa > wb) return 1;
    if (wa < wb) return 0;
    return sa < sb;
}

/* Per row of C logits: the k largest (ties to the lower channel), in the
 * canonical order; S gets their channels and W their logits.  Selection by
 * k passes of "the first not yet taken" (plain, O(k C) per row). */
void moce_oracle_topk(int rows, int C, int k, const double* Lx, int32_t* S, double* W) {
    #pragma omp parallel for schedule(static)
    for (int r = 0; r < rows; ++r) {
        const double* row = Lx + (size_t)r * C;
        unsigned char* taken = (unsigned char*)calloc((size_t)C, 1);
        for (int i = 0; i < k; ++i) {
            int best = -1;
            for (int c = 0; c < C; ++c)
                if (!taken[c] && (best < 0 || comes_before_d(row[c], c, row[best], best))) best = c;
            taken[best] = 1;
            S[(size_t)r * k + i] = best;
            W[(size_t)r * k + i] = row[best];
        }
        free(taken);
    }
}

/* Per example: U(X) = the channels in no support of that example, ascending;
 * U[b][0 .. nU[b]-1]. */
void moce_oracle_dynamic_uncovered(int B, int C, int R, int k, const int32_t* S, int32_t* U, int32_t* nU) {
    #pragma omp parallel for schedule(static)
    for (int b = 0; b < B; ++b) {
        unsigned char* cov = (unsigned char*)calloc((size_t)C, 1);
        for (size_t j = 0; j < (size_t)R * k; ++j) cov[S[(size_t)b * R * k + j]] = 1;
        int n = 0;
        for (int c = 0; c < C; ++c)
            if (!cov[c]) U[(size_t)b * C + n++] = c;
        nU[b] = n;
        free(cov);
    }
}
