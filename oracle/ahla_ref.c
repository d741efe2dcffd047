/*
 * Asymmetric second-order HLA (AHLA, Sec. 6) streaming recurrence in plain C,
 * fp64 (test infrastructure only): Thm. AHLA / Alg. AHLA-stream with decay 1,
 *   P += k_t v_t^T,  m += k_t,  E += k_t (q_t^T P),  n += k_t (q_t^T m),
 *   num_t = q_t^T E,  den_t = q_t^T n.
 * Layouts: q, k [BH, n, d], v [BH, n, dv], num [BH, n, dv], den [BH, n] (may
 * be NULL).  Heads over OpenMP threads.  Returns the number of threads used.
 */
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int ahla_serial_f64(const double *q, const double *k, const double *v, double *num, double *den,
                    long BH, long n, int d, int dv, int nthreads)
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
        double *P = calloc((size_t)d * dv, sizeof(double));
        double *E = calloc((size_t)d * dv, sizeof(double));
        double *m = calloc((size_t)d, sizeof(double));
        double *nn = calloc((size_t)d, sizeof(double));
        double *r = malloc(sizeof(double) * dv);
        for (long t = 0; t < n; ++t) {
            const double *qt = q + (b * n + t) * d;
            const double *kt = k + (b * n + t) * d;
            const double *vt = v + (b * n + t) * dv;
            for (int a = 0; a < d; ++a) {
                for (int j = 0; j < dv; ++j) P[a * dv + j] += kt[a] * vt[j];
                m[a] += kt[a];
            }
            double s = 0.0;
            for (int j = 0; j < dv; ++j) r[j] = 0.0;
            for (int a = 0; a < d; ++a) {
                s += qt[a] * m[a];
                for (int j = 0; j < dv; ++j) r[j] += qt[a] * P[a * dv + j];
            }
            for (int a = 0; a < d; ++a) {
                for (int j = 0; j < dv; ++j) E[a * dv + j] += kt[a] * r[j];
                nn[a] += kt[a] * s;
            }
            double *o = num + (b * n + t) * dv;
            double dd = 0.0;
            for (int j = 0; j < dv; ++j) o[j] = 0.0;
            for (int a = 0; a < d; ++a) {
                dd += qt[a] * nn[a];
                for (int j = 0; j < dv; ++j) o[j] += qt[a] * E[a * dv + j];
            }
            if (den) den[b * n + t] = dd;
        }
        free(P); free(E); free(m); free(nn); free(r);
    }
    return used;
}
