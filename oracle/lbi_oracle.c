/*
 * CPU oracle for the interface-adjoint scan.  TEST INFRASTRUCTURE ONLY:
 * tests, the smoke check and the benchmark's CPU baseline may call it; the
 * product path never does.  It shares no code with the HIP library.
 *
 * Definitions followed (paper: "LBI: Parallel Scan Backpropagation via
 * Latent Bounded Interfaces"):
 *   - Theorem "Bounded-Interface Backpropagation" (Scan Formulation section):
 *     the interface adjoints obey  mbar_k = J_k^T mbar_{k+1},  k = K-1..0,
 *     with J_k = d m_{k+1} / d m_k, and equal the product form
 *     mbar_k = (J_k^T J_{k+1}^T ... J_{K-1}^T) mbar_K  (empty product = I).
 *   - The affine term b_k is the direct gradient of any loss term that reads
 *     m_k; with it the chain rule gives  lambda_k = A_k lambda_{k+1} + b_k,
 *     A_k = J_k^T.  With b = 0 this is exactly the theorem.
 *   - Proposition "Scan Formulation of Backpropagation": the suffix products
 *     P_k = A_k ... A_{K-1} (and, with the affine term, the offsets
 *     c_k = A_k c_{k+1} + b_k, c_K = 0) give lambda_k = P_k lambda_K + c_k.
 *
 * Precision: every input element is widened exactly to double; all sums and
 * products are double.  Built with -ffp-contract=off so that a*x + y is a
 * rounded product followed by a rounded sum, in a fixed order.
 *
 * Layout (row-major): A[beta][j][i][k] = (J_j^T)[i][k], b[beta][j][i],
 * lamK[beta][i], lam[beta][j][i] for j = 0..K-1 (slot K is the input).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_F64 = 0, ORC_F32 = 1, ORC_BF16 = 2 };

static double widen(const void *base, int dtype, int64_t idx)
{
    if (dtype == ORC_F64)
        return ((const double *)base)[idx];
    if (dtype == ORC_F32)
        return (double)((const float *)base)[idx];
    /* bfloat16: the upper 16 bits of an IEEE binary32 */
    uint32_t u = ((uint32_t)((const uint16_t *)base)[idx]) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * lambda_j = A_j lambda_{j+1} + b_j for j = K-1 down to 0 (b may be NULL,
 * meaning b = 0).  One independent chain per beta; chains are shared out over
 * `nthreads` OpenMP threads (<= 0: the OpenMP default).  Returns 0, or -1 on a
 * bad argument.
 */
int lbi_oracle_recurrence(const void *A, const void *b, const void *lamK, double *lam,
                          int64_t B, int64_t K, int32_t r, int dtype, int nthreads)
{
    if (B < 0 || K < 1 || r < 1 || !A || !lamK || !lam)
        return -1;
    if (dtype != ORC_F64 && dtype != ORC_F32 && dtype != ORC_BF16)
        return -1;
#ifdef _OPENMP
    const int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
#endif
    for (int64_t beta = 0; beta < B; ++beta) {
        double *x = (double *)malloc(sizeof(double) * (size_t)r);
        double *y = (double *)malloc(sizeof(double) * (size_t)r);
        for (int32_t i = 0; i < r; ++i)
            x[i] = widen(lamK, dtype, beta * r + i);
        for (int64_t j = K - 1; j >= 0; --j) {
            const int64_t slot = beta * K + j;
            const int64_t abase = slot * (int64_t)r * r;
            for (int32_t i = 0; i < r; ++i) {
                double acc = 0.0;
                for (int32_t k = 0; k < r; ++k)
                    acc += widen(A, dtype, abase + (int64_t)i * r + k) * x[k];
                if (b)
                    acc += widen(b, dtype, slot * r + i);
                y[i] = acc;
            }
            for (int32_t i = 0; i < r; ++i) {
                x[i] = y[i];
                lam[slot * r + i] = y[i];
            }
        }
        free(x);
        free(y);
    }
    (void)nthreads;
    return 0;
}

/* Number of threads the recurrence uses for `nthreads` (<= 0: the default). */
int lbi_oracle_threads(int nthreads)
{
#ifdef _OPENMP
    return nthreads > 0 ? nthreads : omp_get_max_threads();
#else
    (void)nthreads;
    return 1;
#endif
}

/*
 * Suffix composites of the scan: P_j = A_j P_{j+1}, c_j = A_j c_{j+1} + b_j,
 * with P_K = I and c_K = 0, for j = K-1 down to 0.  This is the combine
 * (A, b) o (A', b') = (A A', A b' + b) applied from the right end of the chain,
 * i.e. the inclusive suffix scan of the slots under that combine.
 * Outputs P[beta][j][i][k] and c[beta][j][i] in double.
 */
int lbi_oracle_suffix_composites(const void *A, const void *b, double *P, double *c,
                                 int64_t B, int64_t K, int32_t r, int dtype)
{
    if (B < 0 || K < 1 || r < 1 || !A || !P || !c)
        return -1;
    if (dtype != ORC_F64 && dtype != ORC_F32 && dtype != ORC_BF16)
        return -1;
    const int64_t rr = (int64_t)r * r;
    for (int64_t beta = 0; beta < B; ++beta) {
        for (int64_t j = K - 1; j >= 0; --j) {
            const int64_t slot = beta * K + j;
            double *Pj = P + slot * rr;
            double *cj = c + slot * r;
            const double *Pn = (j == K - 1) ? NULL : P + (slot + 1) * rr;
            const double *cn = (j == K - 1) ? NULL : c + (slot + 1) * r;
            for (int32_t i = 0; i < r; ++i) {
                for (int32_t n = 0; n < r; ++n) {
                    double acc = 0.0;
                    if (Pn) {
                        for (int32_t k = 0; k < r; ++k)
                            acc += widen(A, dtype, slot * rr + (int64_t)i * r + k) * Pn[(int64_t)k * r + n];
                    } else {
                        acc = widen(A, dtype, slot * rr + (int64_t)i * r + n); /* A_{K-1} I */
                    }
                    Pj[(int64_t)i * r + n] = acc;
                }
                double acc = 0.0;
                if (cn)
                    for (int32_t k = 0; k < r; ++k)
                        acc += widen(A, dtype, slot * rr + (int64_t)i * r + k) * cn[k];
                if (b)
                    acc += widen(b, dtype, slot * r + i);
                cj[i] = acc;
            }
        }
    }
    return 0;
}
