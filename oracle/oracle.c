/*
 * CPU oracle for Semidirect Fourier Delta Attention (SFDA) -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg use this
 * file.  It shares no code with the GPU library and must never be linked into it.
 *
 * It evaluates the tied SFDA recurrence token by token in complex double precision,
 * written straight from its definition:
 *
 *   Lambda_t = diag(alpha_t * exp(i theta_t))                 (Sec. 3, Eq. (sfda))
 *   S_t      = (I - beta_t k_t k_t^*) Lambda_t S_{t-1} + beta_t k_t v_t^*
 *   o_t      = S_t^* q_t                                      (readout after the update)
 *
 * where x^* is the conjugate transpose (App. A, block-WY identity over C), so
 * (k v^*)_{ij} = k_i conj(v_j) and o_{t,j} = sum_i conj(S_{ij}) q_i.
 * The update is applied in the order the definition reads: first the phase-decay
 * Lambda_t, then the erase (I - beta k k^*), then the write beta k v^*.
 *
 * Complex numbers are written as explicit (re, im) pairs of doubles so that no
 * library complex routine (and no range-extension path) is involved.
 *
 * Layouts (row-major, complex = interleaved re, im):
 *   q, k   [B,H,T,m,2]    v, o  [B,H,T,n,2]
 *   alpha, theta [B,H,T,m]   beta [B,H,T]
 *   S0, S_T [B,H,m,n,2]  (S0 == NULL means the zero state)
 * Heads (b, h) are independent; they are spread over OpenMP threads.
 */
#include <math.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* One head, T tokens.  S (m x n complex) is updated in place. */
static void sfda_head(int T, int m, int n,
                      const double* q, const double* k, const double* v,
                      const double* alpha, const double* theta, const double* beta,
                      double* S, double* o, double* x /* scratch, 2n */)
{
    for (int t = 0; t < T; ++t) {
        const double* qt = q + (size_t)t * m * 2;
        const double* kt = k + (size_t)t * m * 2;
        const double* vt = v + (size_t)t * n * 2;
        const double* at = alpha + (size_t)t * m;
        const double* th = theta + (size_t)t * m;
        const double bt = beta[t];

        /* S <- Lambda_t S : row i is multiplied by lambda_i = alpha_i (cos theta_i + i sin theta_i) */
        for (int i = 0; i < m; ++i) {
            const double lr = at[i] * cos(th[i]);
            const double li = at[i] * sin(th[i]);
            double* row = S + (size_t)i * n * 2;
            for (int j = 0; j < n; ++j) {
                const double sr = row[2 * j], si = row[2 * j + 1];
                row[2 * j] = lr * sr - li * si;
                row[2 * j + 1] = lr * si + li * sr;
            }
        }
        /* x = k_t^* (Lambda_t S) : x_j = sum_i conj(k_i) S_ij */
        for (int j = 0; j < 2 * n; ++j) x[j] = 0.0;
        for (int i = 0; i < m; ++i) {
            const double kr = kt[2 * i], ki = kt[2 * i + 1];
            const double* row = S + (size_t)i * n * 2;
            for (int j = 0; j < n; ++j) {
                const double sr = row[2 * j], si = row[2 * j + 1];
                x[2 * j] += kr * sr + ki * si;
                x[2 * j + 1] += kr * si - ki * sr;
            }
        }
        /* S <- S - beta k x + beta k v^*  =  S + beta k (conj(v) - x)  (row i gets k_i times it) */
        for (int j = 0; j < n; ++j) {
            x[2 * j] = bt * (vt[2 * j] - x[2 * j]);
            x[2 * j + 1] = bt * (-vt[2 * j + 1] - x[2 * j + 1]);
        }
        for (int i = 0; i < m; ++i) {
            const double kr = kt[2 * i], ki = kt[2 * i + 1];
            double* row = S + (size_t)i * n * 2;
            for (int j = 0; j < n; ++j) {
                const double dr = x[2 * j], di = x[2 * j + 1];
                row[2 * j] += kr * dr - ki * di;
                row[2 * j + 1] += kr * di + ki * dr;
            }
        }
        /* o_t = S_t^* q_t : o_j = sum_i conj(S_ij) q_i */
        double* ot = o + (size_t)t * n * 2;
        for (int j = 0; j < 2 * n; ++j) ot[j] = 0.0;
        for (int i = 0; i < m; ++i) {
            const double qr = qt[2 * i], qi = qt[2 * i + 1];
            const double* row = S + (size_t)i * n * 2;
            for (int j = 0; j < n; ++j) {
                const double sr = row[2 * j], si = row[2 * j + 1];
                ot[2 * j] += sr * qr + si * qi;
                ot[2 * j + 1] += sr * qi - si * qr;
            }
        }
    }
}

/* Full forward: o for every token and the state after the last token.
 * Returns 0 on success, 1 on bad arguments, 2 on allocation failure.
 * nthreads <= 0 uses the OpenMP default. */
int oracle_recurrence(int B, int H, int T, int m, int n,
                      const double* q, const double* k, const double* v,
                      const double* alpha, const double* theta, const double* beta,
                      const double* S0, double* o, double* S_T, int nthreads)
{
    if (B < 0 || H < 0 || T < 0 || m <= 0 || n <= 0) return 1;
    if (!q || !k || !v || !alpha || !theta || !beta || !o || !S_T) return 1;
    const long heads = (long)B * H;
    int err = 0;
#ifdef _OPENMP
    if (nthreads <= 0) nthreads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads) reduction(|: err)
#endif
    for (long bh = 0; bh < heads; ++bh) {
        double* x = (double*)malloc(sizeof(double) * 2 * n);
        if (!x) { err |= 2; continue; }
        double* S = S_T + (size_t)bh * m * n * 2;
        if (S0) memmove(S, S0 + (size_t)bh * m * n * 2, sizeof(double) * 2 * m * n);
        else memset(S, 0, sizeof(double) * 2 * m * n);
        sfda_head(T, m, n,
                  q + (size_t)bh * T * m * 2, k + (size_t)bh * T * m * 2,
                  v + (size_t)bh * T * n * 2, alpha + (size_t)bh * T * m,
                  theta + (size_t)bh * T * m, beta + (size_t)bh * T,
                  S, o + (size_t)bh * T * n * 2, x);
        free(x);
    }
    return err;
}

/* One decode token for every head: S [B,H,m,n,2] updated in place, o [B,H,n,2].
 * Inputs q,k [B,H,m,2], v [B,H,n,2], alpha,theta [B,H,m], beta [B,H]. */
int oracle_step(int B, int H, int m, int n,
                const double* q, const double* k, const double* v,
                const double* alpha, const double* theta, const double* beta,
                double* S, double* o, int nthreads)
{
    if (B < 0 || H < 0 || m <= 0 || n <= 0) return 1;
    if (!q || !k || !v || !alpha || !theta || !beta || !S || !o) return 1;
    const long heads = (long)B * H;
    int err = 0;
#ifdef _OPENMP
    if (nthreads <= 0) nthreads = omp_get_max_threads();
#pragma omp parallel for schedule(static) num_threads(nthreads) reduction(|: err)
#endif
    for (long bh = 0; bh < heads; ++bh) {
        double* x = (double*)malloc(sizeof(double) * 2 * n);
        if (!x) { err |= 2; continue; }
        sfda_head(1, m, n, q + (size_t)bh * m * 2, k + (size_t)bh * m * 2,
                  v + (size_t)bh * n * 2, alpha + (size_t)bh * m, theta + (size_t)bh * m,
                  beta + bh, S + (size_t)bh * m * n * 2, o + (size_t)bh * n * 2, x);
        free(x);
    }
    return err;
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
