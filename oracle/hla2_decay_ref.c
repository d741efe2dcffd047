/*
 * Second-order HLA with exponential decay, serial recurrence in plain C, fp64
 * (test infrastructure only).  The recurrence of the decayed module of this
 * oracle (decayed moments of the decay section; cross-summaries read so that
 * the masked output is the unmasked decayed output with the pairs j < i
 * removed at the same weights gamma^{(t-i)+(t-j)}):
 *   G = g^2 G + g k_t (k_t^T C_{t-1}),  h = g^2 h + g k_t (k_t^T m_{t-1}),
 *   S = g S + k_t k_t^T,  C = g C + q_t v_t^T,  m = g m + q_t,
 * then the Thm. 1 readout (u = q^T S, num = u C - q^T G, den = u m - q^T h).
 * Layouts and the state arguments are those of hla2_serial_f64; heads over
 * OpenMP threads.  Returns the number of threads used.
 */
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int hla2_decay_serial_f64(const double *q, const double *k, const double *v,
                          double *num, double *den,
                          long BH, long n, int d, int dv, int masked, double gamma,
                          double *state_S, double *state_C, double *state_m,
                          double *state_G, double *state_h, int nthreads)
{
    int used = 1;
    const double g = gamma, g2 = gamma * gamma;
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
            double s = 0.0;                       /* k_t^T m_{t-1} */
            for (int j = 0; j < dv; ++j) w[j] = 0.0;
            for (int a = 0; a < d; ++a) {
                s += kt[a] * m[a];
                for (int j = 0; j < dv; ++j) w[j] += kt[a] * C[a * dv + j];   /* k_t^T C_{t-1} */
            }
            for (int a = 0; a < d; ++a) {
                for (int j = 0; j < dv; ++j) G[a * dv + j] = g2 * G[a * dv + j] + g * kt[a] * w[j];
                h[a] = g2 * h[a] + g * s * kt[a];
                for (int c = 0; c < d; ++c) S[a * d + c] = g * S[a * d + c] + kt[a] * kt[c];
                for (int j = 0; j < dv; ++j) C[a * dv + j] = g * C[a * dv + j] + qt[a] * vt[j];
                m[a] = g * m[a] + qt[a];
            }
            for (int c = 0; c < d; ++c) u[c] = 0.0;
            for (int a = 0; a < d; ++a)
                for (int c = 0; c < d; ++c) u[c] += qt[a] * S[a * d + c];
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
