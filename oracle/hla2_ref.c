/*
 * Second-order HLA oracle in plain C, fp64 (test infrastructure only).
 *
 * The serial left-to-right recurrence of the paper: the online updates of
 * Sec. 3.1 followed by the readout of Thm. 1 in the order of Sec. 5
 * (u = q^T S, num = u C - q^T G, den = u m - q^T h).  Decay 1, ridge 0.
 * Heads are independent (Sec. 5.2) and are spread over OpenMP threads.
 *
 * Layouts (row-major, contiguous, BH = number of independent heads):
 *   q, k  [BH, n, d]     v  [BH, n, dv]     num [BH, n, dv]    den [BH, n]
 *   state: S [BH, d, d], C [BH, d, dv], m [BH, d], G [BH, d, dv], h [BH, d]
 * `state_*` arrays hold the initial state on entry (NULL = zero state) and the
 * final state on exit (NULL = not returned).  `den` may be NULL.
 * `masked` = 0 gives the unmasked operator q^T S C (and q^T S m).
 * Returns the number of threads used.
 */
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int hla2_serial_f64(const double *q, const double *k, const double *v,
                    double *num, double *den,
                    long BH, long n, int d, int dv, int masked,
                    double *state_S, double *state_C, double *state_m,
                    double *state_G, double *state_h, int nthreads)
{
    int used = 1;
#ifdef _OPENMP
    if (nthreads <= 0) nthreads = omp_get_max_threads();
    if (nthreads > BH) nthreads = (int)BH;
    if (nthreads < 1) nthreads = 1;
    used = nthreads;
#pragma omp parallel for num_threads(nthreads) schedule(dynamic, 1)
#endif
    for (long b = 0; b < BH; ++b) {
        double *S = calloc((size_t)d * d, sizeof(double));
        double *C = calloc((size_t)d * dv, sizeof(double));
        double *G = calloc((size_t)d * dv, sizeof(double));
        double *m = calloc((size_t)d, sizeof(double));
        double *h = calloc((size_t)d, sizeof(double));
        double *w = malloc(sizeof(double) * dv);
        double *u = malloc(sizeof(double) * d);
        if (state_S) memcpy(S, state_S + b * d * d, sizeof(double) * d * d);
        if (state_C) memcpy(C, state_C + b * d * dv, sizeof(double) * d * dv);
        if (state_m) memcpy(m, state_m + b * d, sizeof(double) * d);
        if (state_G) memcpy(G, state_G + b * d * dv, sizeof(double) * d * dv);
        if (state_h) memcpy(h, state_h + b * d, sizeof(double) * d);
        for (long t = 0; t < n; ++t) {
            const double *qt = q + (b * n + t) * d;
            const double *kt = k + (b * n + t) * d;
            const double *vt = v + (b * n + t) * dv;
            /* w = k_t^T C_{t-1},  s = k_t^T m_{t-1} */
            double s = 0.0;
            for (int j = 0; j < dv; ++j) w[j] = 0.0;
            for (int a = 0; a < d; ++a) {
                s += kt[a] * m[a];
                for (int j = 0; j < dv; ++j) w[j] += kt[a] * C[a * dv + j];
            }
            /* G += k_t w^T, h += s k_t, S += k_t k_t^T, C += q_t v_t^T, m += q_t */
            for (int a = 0; a < d; ++a) {
                for (int j = 0; j < dv; ++j) G[a * dv + j] += kt[a] * w[j];
                h[a] += s * kt[a];
                for (int c = 0; c < d; ++c) S[a * d + c] += kt[a] * kt[c];
                for (int j = 0; j < dv; ++j) C[a * dv + j] += qt[a] * vt[j];
                m[a] += qt[a];
            }
            /* u = q_t^T S_t */
            for (int c = 0; c < d; ++c) u[c] = 0.0;
            for (int a = 0; a < d; ++a)
                for (int c = 0; c < d; ++c) u[c] += qt[a] * S[a * d + c];
            /* num = u C_t - q_t^T G_t,  den = u m_t - q_t^T h_t */
            double *nt = num + (b * n + t) * dv;
            double dt = 0.0;
            for (int j = 0; j < dv; ++j) nt[j] = 0.0;
            for (int a = 0; a < d; ++a) {
                dt += u[a] * m[a];
                if (masked) dt -= qt[a] * h[a];
                for (int j = 0; j < dv; ++j) {
                    nt[j] += u[a] * C[a * dv + j];
                    if (masked) nt[j] -= qt[a] * G[a * dv + j];
                }
            }
            if (den) den[b * n + t] = dt;
        }
        if (state_S) memcpy(state_S + b * d * d, S, sizeof(double) * d * d);
        if (state_C) memcpy(state_C + b * d * dv, C, sizeof(double) * d * dv);
        if (state_m) memcpy(state_m + b * d, m, sizeof(double) * d);
        if (state_G) memcpy(state_G + b * d * dv, G, sizeof(double) * d * dv);
        if (state_h) memcpy(state_h + b * d, h, sizeof(double) * d);
        free(S); free(C); free(G); free(m); free(h); free(w); free(u);
    }
    return used;
}
