/*
 * The C oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
 * (tests/test_oracle_sanitize.py compiles and runs this), exercised over its
 * whole interface: every input dtype, with and without b, several thread
 * counts, the suffix composites, and the argument checks.  Values are checked
 * against facts that do not come from the oracle:
 *   - small-integer inputs: the product form of Theorem "Bounded-Interface
 *     Backpropagation" (lambda_j = (A_j ... A_{K-1}) lambda_K + sum_i
 *     (A_j ... A_{i-1}) b_i), formed here in exact 64-bit integer arithmetic;
 *     every value is far below 2^53, so the fp64 oracle must equal it;
 *   - the suffix composites P_j, c_j against the same integer products;
 *   - A = I, b = 0: lambda_j = lambda_K for float32 and bfloat16 storage;
 *   - results bit for bit the same for 1, 2 and 5 threads.
 * Exit status 0 when every check passes; a sanitizer report aborts.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../oracle/lbi_oracle.c"

static int failures = 0;
#define CHECK(cond, ...)                        \
    do {                                        \
        if (!(cond)) {                          \
            fprintf(stderr, "FAIL: " __VA_ARGS__); \
            fprintf(stderr, "\n");              \
            ++failures;                         \
        }                                       \
    } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static int small_int(void) /* uniform in [-3, 3], splitmix64 */
{
    uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    return (int)(z % 7) - 3;
}

/* exact integer suffix products and adjoints of one chain */
static void integer_reference(const int64_t *A, const int64_t *b, const int64_t *lk, int64_t K,
                              int r, int64_t *P, int64_t *c, int64_t *lam)
{
    for (int64_t j = K - 1; j >= 0; --j) {
        const int64_t *Aj = A + j * r * r;
        int64_t *Pj = P + j * r * r, *cj = c + j * r;
        for (int i = 0; i < r; ++i) {
            for (int n = 0; n < r; ++n) {
                int64_t acc = 0;
                if (j == K - 1)
                    acc = Aj[i * r + n];
                else
                    for (int k = 0; k < r; ++k)
                        acc += Aj[i * r + k] * P[(j + 1) * r * r + k * r + n];
                Pj[i * r + n] = acc;
            }
            int64_t acc = b ? b[j * r + i] : 0;
            if (j < K - 1)
                for (int k = 0; k < r; ++k)
                    acc += Aj[i * r + k] * c[(j + 1) * r + k];
            cj[i] = acc;
        }
        for (int i = 0; i < r; ++i) {
            int64_t acc = cj[i];
            for (int k = 0; k < r; ++k)
                acc += Pj[i * r + k] * lk[k];
            lam[j * r + i] = acc;
        }
    }
}

static uint16_t bf16_of_int(int v) /* small integers are exact in bfloat16 */
{
    float f = (float)v;
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return (uint16_t)(u >> 16);
}

static void integer_case(int64_t B, int64_t K, int r, int affine)
{
    const int64_t nA = B * K * r * r, nb = B * K * r, nl = B * r;
    int64_t *Ai = malloc(sizeof(int64_t) * nA), *bi = malloc(sizeof(int64_t) * nb);
    int64_t *li = malloc(sizeof(int64_t) * nl);
    double *Ad = malloc(sizeof(double) * nA), *bd = malloc(sizeof(double) * nb);
    double *ld = malloc(sizeof(double) * nl);
    float *Af = malloc(sizeof(float) * nA), *bf = malloc(sizeof(float) * nb);
    float *lf = malloc(sizeof(float) * nl);
    uint16_t *Ah = malloc(sizeof(uint16_t) * nA), *bh = malloc(sizeof(uint16_t) * nb);
    uint16_t *lh = malloc(sizeof(uint16_t) * nl);
    for (int64_t i = 0; i < nA; ++i) {
        Ai[i] = small_int();
        Ad[i] = (double)Ai[i];
        Af[i] = (float)Ai[i];
        Ah[i] = bf16_of_int((int)Ai[i]);
    }
    for (int64_t i = 0; i < nb; ++i) {
        bi[i] = small_int();
        bd[i] = (double)bi[i];
        bf[i] = (float)bi[i];
        bh[i] = bf16_of_int((int)bi[i]);
    }
    for (int64_t i = 0; i < nl; ++i) {
        li[i] = small_int();
        ld[i] = (double)li[i];
        lf[i] = (float)li[i];
        lh[i] = bf16_of_int((int)li[i]);
    }
    int64_t *P = malloc(sizeof(int64_t) * K * r * r), *c = malloc(sizeof(int64_t) * K * r);
    int64_t *want = malloc(sizeof(int64_t) * nb);
    for (int64_t beta = 0; beta < B; ++beta)
        integer_reference(Ai + beta * K * r * r, affine ? bi + beta * K * r : NULL, li + beta * r,
                          K, r, P, c, want + beta * K * r);
    const void *As[3] = {Ad, Af, Ah}, *bs[3] = {bd, bf, bh}, *ls[3] = {ld, lf, lh};
    double *lam = malloc(sizeof(double) * nb), *lam1 = malloc(sizeof(double) * nb);
    for (int dt = 0; dt < 3; ++dt) {
        for (int nt = 1; nt <= 5; nt += 2) {
            CHECK(lbi_oracle_recurrence(As[dt], affine ? bs[dt] : NULL, ls[dt], lam, B, K, r, dt,
                                        nt) == 0,
                  "recurrence rejected valid arguments");
            for (int64_t i = 0; i < nb; ++i)
                CHECK(lam[i] == (double)want[i], "dtype %d threads %d: lam[%lld] = %g, want %lld",
                      dt, nt, (long long)i, lam[i], (long long)want[i]);
            if (nt == 1)
                memcpy(lam1, lam, sizeof(double) * nb);
            else
                CHECK(memcmp(lam, lam1, sizeof(double) * nb) == 0, "thread count changed bits");
        }
    }
    /* the suffix composites of every chain */
    double *Pd = malloc(sizeof(double) * nA), *cd = malloc(sizeof(double) * nb);
    CHECK(lbi_oracle_suffix_composites(Ad, affine ? bd : NULL, Pd, cd, B, K, r, ORC_F64) == 0,
          "composites rejected valid arguments");
    for (int64_t beta = 0; beta < B; ++beta) {
        integer_reference(Ai + beta * K * r * r, affine ? bi + beta * K * r : NULL, li + beta * r,
                          K, r, P, c, want);
        for (int64_t i = 0; i < K * r * r; ++i)
            CHECK(Pd[beta * K * r * r + i] == (double)P[i], "P mismatch at chain %lld",
                  (long long)beta);
        for (int64_t i = 0; i < K * r; ++i)
            CHECK(cd[beta * K * r + i] == (double)c[i], "c mismatch at chain %lld",
                  (long long)beta);
    }
    free(Ai); free(bi); free(li); free(Ad); free(bd); free(ld); free(Af); free(bf); free(lf);
    free(Ah); free(bh); free(lh); free(P); free(c); free(want); free(lam); free(lam1);
    free(Pd); free(cd);
}

static void identity_case(void)
{
    const int64_t B = 2, K = 9;
    const int r = 16;
    float *A = calloc((size_t)(B * K * r * r), sizeof(float));
    uint16_t *Ah = calloc((size_t)(B * K * r * r), sizeof(uint16_t));
    float *lk = malloc(sizeof(float) * B * r);
    uint16_t *lkh = malloc(sizeof(uint16_t) * B * r);
    for (int64_t s = 0; s < B * K; ++s)
        for (int i = 0; i < r; ++i) {
            A[s * r * r + i * r + i] = 1.0f;
            Ah[s * r * r + i * r + i] = bf16_of_int(1);
        }
    for (int64_t i = 0; i < B * r; ++i) {
        lk[i] = (float)small_int() * 0.25f;  /* exact in both storages */
        uint32_t u;
        memcpy(&u, &lk[i], sizeof u);
        lkh[i] = (uint16_t)(u >> 16);
    }
    double *lam = malloc(sizeof(double) * B * K * r);
    CHECK(lbi_oracle_recurrence(A, NULL, lk, lam, B, K, r, ORC_F32, 2) == 0, "identity f32");
    for (int64_t beta = 0; beta < B; ++beta)
        for (int64_t j = 0; j < K; ++j)
            for (int i = 0; i < r; ++i)
                CHECK(lam[(beta * K + j) * r + i] == (double)lk[beta * r + i], "identity f32");
    CHECK(lbi_oracle_recurrence(Ah, NULL, lkh, lam, B, K, r, ORC_BF16, 3) == 0, "identity bf16");
    for (int64_t beta = 0; beta < B; ++beta)
        for (int64_t j = 0; j < K; ++j)
            for (int i = 0; i < r; ++i)
                CHECK(lam[(beta * K + j) * r + i] == (double)lk[beta * r + i], "identity bf16");
    free(A); free(Ah); free(lk); free(lkh); free(lam);
}

static void argument_checks(void)
{
    double a[16] = {0}, l[4] = {0}, out[64];
    CHECK(lbi_oracle_recurrence(a, NULL, l, out, -1, 1, 4, ORC_F64, 1) == -1, "B < 0");
    CHECK(lbi_oracle_recurrence(a, NULL, l, out, 1, 0, 4, ORC_F64, 1) == -1, "K < 1");
    CHECK(lbi_oracle_recurrence(a, NULL, l, out, 1, 1, 0, ORC_F64, 1) == -1, "r < 1");
    CHECK(lbi_oracle_recurrence(NULL, NULL, l, out, 1, 1, 4, ORC_F64, 1) == -1, "NULL A");
    CHECK(lbi_oracle_recurrence(a, NULL, l, out, 1, 1, 4, 7, 1) == -1, "bad dtype");
    CHECK(lbi_oracle_suffix_composites(a, NULL, NULL, out, 1, 1, 4, ORC_F64) == -1, "NULL P");
    CHECK(lbi_oracle_recurrence(a, NULL, l, out, 0, 1, 4, ORC_F64, 1) == 0, "B = 0 no-op");
    CHECK(lbi_oracle_threads(3) == 3 || lbi_oracle_threads(3) == 1, "threads");
}

int main(void)
{
    integer_case(3, 5, 4, 1);
    integer_case(2, 6, 3, 0);
    integer_case(4, 1, 2, 1);
    integer_case(5, 4, 5, 1);
    identity_case();
    argument_checks();
    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("oracle sanitizer run: all checks passed\n");
    return 0;
}
