/*
 * Third-order HLA oracle in plain C, fp64 (test infrastructure only).
 *
 * Alg. 3 (Sec. 7.2) with decay 1: per token, with the moments before it
 * (SK', SQ', P', m'), the inclusive moments SK, SQ, P, m, the corrections
 *   G1 += k ((SQ' k)^T P'),  h1 += k ((SQ' k) . m')
 *   G2 += (SK' q)(q^T P'),   h2 += (SK' q)(q . m')
 *   G3 += (SK' SQ' k) v^T,   h3 += SK' SQ' k
 * and the readout num = (SQ SK q)^T P - q^T (G1 + G2 + G3),
 * den = (SQ SK q) . m - q . (h1 + h2 + h3) (Thm. 3); masked = 0 keeps only
 * the first terms.  Heads are independent and spread over OpenMP threads.
 *
 * Layouts (row-major, contiguous): q, k [BH, n, d], v [BH, n, dv],
 * num [BH, n, dv], den [BH, n] (den may be NULL).  Returns the number of
 * threads used.
 */
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int hla3_serial_f64(const double *q, const double *k, const double *v,
                    double *num, double *den,
                    long BH, long n, int d, int dv, int masked, int nthreads)
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
        const size_t dd = (size_t)d * d, ddv = (size_t)d * dv;
        double *SK = calloc(dd, sizeof(double)), *SQ = calloc(dd, sizeof(double));
        double *P = calloc(ddv, sizeof(double)), *G = calloc(ddv, sizeof(double));
        double *m = calloc(d, sizeof(double)), *hs = calloc(d, sizeof(double));
        double *u1 = malloc(d * sizeof(double)), *a2 = malloc(d * sizeof(double));
        double *a3 = malloc(d * sizeof(double)), *y = malloc(d * sizeof(double));
        double *z = malloc(d * sizeof(double)), *r1 = malloc(dv * sizeof(double));
        double *r2 = malloc(dv * sizeof(double));
        for (long t = 0; t < n; ++t) {
            const double *qt = q + ((size_t)b * n + t) * d;
            const double *kt = k + ((size_t)b * n + t) * d;
            const double *vt = v + ((size_t)b * n + t) * dv;
            /* corrections from the moments before token t (G = G1 + G2 + G3, hs = h1 + h2 + h3) */
            double s1 = 0.0, s2 = 0.0;
            for (int a = 0; a < d; ++a) {
                double x = 0.0, w = 0.0;
                for (int c = 0; c < d; ++c) {
                    x += SQ[(size_t)a * d + c] * kt[c];     /* u1 = SQ' k */
                    w += SK[(size_t)a * d + c] * qt[c];     /* a2 = SK' q */
                }
                u1[a] = x;
                a2[a] = w;
            }
            for (int a = 0; a < d; ++a) {
                double x = 0.0;
                for (int c = 0; c < d; ++c) x += SK[(size_t)a * d + c] * u1[c];   /* a3 = SK' SQ' k */
                a3[a] = x;
                s1 += u1[a] * m[a];
                s2 += qt[a] * m[a];
            }
            for (int e = 0; e < dv; ++e) {
                double x = 0.0, w = 0.0;
                for (int a = 0; a < d; ++a) {
                    x += u1[a] * P[(size_t)a * dv + e];     /* u1^T P' */
                    w += qt[a] * P[(size_t)a * dv + e];     /* q^T P'  */
                }
                r1[e] = x;
                r2[e] = w;
            }
            for (int a = 0; a < d; ++a) {
                for (int e = 0; e < dv; ++e)
                    G[(size_t)a * dv + e] += kt[a] * r1[e] + a2[a] * r2[e] + a3[a] * vt[e];
                hs[a] += kt[a] * s1 + a2[a] * s2 + a3[a];
            }
            /* inclusive moments */
            for (int a = 0; a < d; ++a) {
                for (int c = 0; c < d; ++c) {
                    SK[(size_t)a * d + c] += kt[a] * kt[c];
                    SQ[(size_t)a * d + c] += qt[a] * qt[c];
                }
                for (int e = 0; e < dv; ++e) P[(size_t)a * dv + e] += kt[a] * vt[e];
                m[a] += kt[a];
            }
            /* readout: z = SQ SK q */
            for (int a = 0; a < d; ++a) {
                double x = 0.0;
                for (int c = 0; c < d; ++c) x += SK[(size_t)a * d + c] * qt[c];
                y[a] = x;
            }
            for (int a = 0; a < d; ++a) {
                double x = 0.0;
                for (int c = 0; c < d; ++c) x += SQ[(size_t)a * d + c] * y[c];
                z[a] = x;
            }
            double *nt = num + ((size_t)b * n + t) * dv;
            for (int e = 0; e < dv; ++e) {
                double x = 0.0;
                for (int a = 0; a < d; ++a) {
                    x += z[a] * P[(size_t)a * dv + e];
                    if (masked) x -= qt[a] * G[(size_t)a * dv + e];
                }
                nt[e] = x;
            }
            if (den) {
                double x = 0.0;
                for (int a = 0; a < d; ++a) {
                    x += z[a] * m[a];
                    if (masked) x -= qt[a] * hs[a];
                }
                den[(size_t)b * n + t] = x;
            }
        }
        free(SK); free(SQ); free(P); free(G); free(m); free(hs);
        free(u1); free(a2); free(a3); free(y); free(z); free(r1); free(r2);
    }
    return used;
}
