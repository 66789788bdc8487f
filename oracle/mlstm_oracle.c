/*
 * mLSTM cell oracle, recurrent form, fp64, plain C.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct CPU
 * reference that the HIP path is checked against.  Only the tests, the smoke
 * check and the benchmark's CPU-baseline leg may load it; the product path
 * never does.  It shares no code, header or constant with the HIP library.
 *
 * It follows the recurrent ("generation mode") statement of the cell in
 * Sec. 2 of the paper, Eqs. 2-5 with the gate activations of Eqs. 7-8:
 *
 *   m_t = max(logsig(f~_t) + m_{t-1}, i~_t)                        (Eq. 2)
 *   f_t = exp(logsig(f~_t) + m_{t-1} - m_t),  i_t = exp(i~_t - m_t) (Eqs. 7, 8)
 *   C_t = f_t C_{t-1} + i_t k_t v_t^T                               (Eq. 3)
 *   n_t = f_t n_{t-1} + i_t k_t                                     (Eq. 4)
 *   h~_t = C_t^T q^_t / max(|n_t^T q^_t|, exp(-m_t)),  q^ = q/sqrt(dqk)  (Eq. 5)
 *
 * Scope: h~ (Eq. 5) and the state; the output gate and Norm of Eq. 6 are
 * not part of the cell computed here.  The zero initial state has m_0 = 0.
 * log sigmoid is evaluated as min(x, 0) - log1p(exp(-|x|)), which is exact
 * in value and does not overflow for large |x|.
 *
 * Parallel over the B*NH independent (batch, head) sequences only; the time
 * loop is sequential.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

static double logsigmoid(double x) { return fmin(x, 0.0) - log1p(exp(-fabs(x))); }

/*
 * q, k: [S, T, DQK]; v: [S, T, DV]; ipre, fpre: [S, T]  with S = B*NH, all fp64.
 * C0: [S, DQK, DV], n0: [S, DQK], m0: [S] or all three NULL (zero state, m0 = 0).
 * h: [S, T, DV]; CT: [S, DQK, DV]; nT: [S, DQK]; mT: [S].
 * Returns 0, or -1 on a bad argument (C0/n0/m0 partially given, negative size).
 */
int oracle_mlstm_recurrent_f64(const double* q, const double* k, const double* v,
                               const double* ipre, const double* fpre,
                               const double* C0, const double* n0, const double* m0,
                               int64_t S, int64_t T, int64_t DQK, int64_t DV,
                               double* h, double* CT, double* nT, double* mT, int nthreads) {
    if (S < 0 || T < 0 || DQK <= 0 || DV <= 0) return -1;
    int have0 = (C0 != NULL) + (n0 != NULL) + (m0 != NULL);
    if (have0 != 0 && have0 != 3) return -1;
    if (nthreads < 1) nthreads = 1;
    const double qscale = 1.0 / sqrt((double)DQK);

#pragma omp parallel num_threads(nthreads)
    {
        double* qh = (double*)malloc(sizeof(double) * (size_t)DQK);
        double* num = (double*)malloc(sizeof(double) * (size_t)DV);
#pragma omp for schedule(dynamic, 1)
        for (int64_t s = 0; s < S; ++s) {
            double* C = CT + s * DQK * DV;
            double* n = nT + s * DQK;
            double m;
            if (have0) {
                memcpy(C, C0 + s * DQK * DV, sizeof(double) * (size_t)(DQK * DV));
                memcpy(n, n0 + s * DQK, sizeof(double) * (size_t)DQK);
                m = m0[s];
            } else {
                memset(C, 0, sizeof(double) * (size_t)(DQK * DV));
                memset(n, 0, sizeof(double) * (size_t)DQK);
                m = 0.0;
            }
            for (int64_t t = 0; t < T; ++t) {
                const double* qt = q + (s * T + t) * DQK;
                const double* kt = k + (s * T + t) * DQK;
                const double* vt = v + (s * T + t) * DV;
                const double a = logsigmoid(fpre[s * T + t]);
                const double it = ipre[s * T + t];
                const double mnew = fmax(a + m, it);
                const double fg = exp(a + m - mnew);
                const double ig = exp(it - mnew);
                for (int64_t d = 0; d < DQK; ++d) {
                    double* Crow = C + d * DV;
                    const double ik = ig * kt[d];
                    for (int64_t j = 0; j < DV; ++j) Crow[j] = fg * Crow[j] + ik * vt[j];
                    n[d] = fg * n[d] + ig * kt[d];
                }
                m = mnew;
                double qn = 0.0;
                for (int64_t d = 0; d < DQK; ++d) {
                    qh[d] = qt[d] * qscale;
                    qn += n[d] * qh[d];
                }
                for (int64_t j = 0; j < DV; ++j) num[j] = 0.0;
                for (int64_t d = 0; d < DQK; ++d) {
                    const double* Crow = C + d * DV;
                    const double qd = qh[d];
                    for (int64_t j = 0; j < DV; ++j) num[j] += Crow[j] * qd;
                }
                const double den = fmax(fabs(qn), exp(-m));
                double* ht = h + (s * T + t) * DV;
                for (int64_t j = 0; j < DV; ++j) ht[j] = num[j] / den;
            }
            mT[s] = m;
        }
        free(qh);
        free(num);
    }
    return 0;
}

int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
