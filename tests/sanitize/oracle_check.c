/*
 * The CPU fp64 oracles (oracle/gmlp_oracle.c, oracle/softmax_matmul_oracle.c)
 * run under AddressSanitizer and UndefinedBehaviorSanitizer: every entry
 * point on small inputs, with row lists (none, explicit, repeated), every
 * activation with and without RMSNorm, one and several threads, empty row
 * lists and the error returns.  Checks a hand-computed example and that
 * results do not depend on the row list or the thread count; exits non-zero
 * on a mismatch (a sanitizer report aborts the run).
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int gmlp_oracle_variant_rows_f64(const double *X, const double *Wg, const double *Wu, const double *Wd,
                                 int64_t T, int64_t D, int64_t F, int act, double beta, int rms, double eps,
                                 const int64_t *rows, int64_t n, double *Y, double *H, int threads);
int gmlp_oracle_variant_rows_bf16(const uint16_t *X, const uint16_t *Wg, const uint16_t *Wu,
                                  const uint16_t *Wd, int64_t T, int64_t D, int64_t F, int act, double beta,
                                  int rms, double eps, const int64_t *rows, int64_t n, double *Y, double *H,
                                  int threads);
int gmlp_oracle_rows_f64(const double *X, const double *Wg, const double *Wu, const double *Wd, int64_t T,
                         int64_t D, int64_t F, const int64_t *rows, int64_t n, double *Y, double *H, int threads);
int gmlp_oracle_down_rows_bf16(const uint16_t *H, const uint16_t *Wd, int64_t T, int64_t F, int64_t D,
                               const int64_t *rows, int64_t n, double *Y, int threads);
int smm_oracle_rows_f64(const double *X, const double *Y, int64_t M, int64_t K, int64_t N, const int64_t *rows,
                        int64_t n, double *Z, double *A, int threads);
int smm_oracle_rows_bf16(const uint16_t *X, const uint16_t *Y, int64_t M, int64_t K, int64_t N,
                         const int64_t *rows, int64_t n, double *Z, double *A, int threads);

static int failures;

#define EXPECT(cond)                                                        \
    do {                                                                    \
        if (!(cond)) {                                                      \
            fprintf(stderr, "FAILED %s:%d: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                     \
        }                                                                   \
    } while (0)

static uint64_t state = 88172645463325252ull;
static double uniform(void) /* xorshift64, in [-1, 1) */
{
    state ^= state << 13;
    state ^= state >> 7;
    state ^= state << 17;
    return (double)(state >> 11) / (double)(1ull << 52) - 1.0;
}

static void fill(double *a, size_t n, double scale)
{
    for (size_t i = 0; i < n; ++i)
        a[i] = scale * uniform();
}

/* bf16 bits of a double, by truncation of its binary32 value (any bf16 will do). */
static void fill_bf16(uint16_t *a, size_t n, double scale)
{
    for (size_t i = 0; i < n; ++i) {
        float f = (float)(scale * uniform());
        uint32_t u;
        memcpy(&u, &f, 4);
        a[i] = (uint16_t)(u >> 16);
    }
}

static int same(const double *a, const double *b, size_t n)
{
    return memcmp(a, b, n * sizeof(double)) == 0;
}

int main(void)
{
    /* Hand-computed example: X = [1, 2], Wg = I, Wu = ones, Wd = [[1, 2], [3, 4]]. */
    {
        const double X[2] = {1, 2}, Wg[4] = {1, 0, 0, 1}, Wu[4] = {1, 1, 1, 1}, Wd[4] = {1, 2, 3, 4};
        double Y[2], H[2];
        EXPECT(gmlp_oracle_rows_f64(X, Wg, Wu, Wd, 1, 2, 2, NULL, 1, Y, H, 1) == 0);
        EXPECT(fabs(Y[0] - 18.047523139491897) < 1e-12 && fabs(Y[1] - 25.525481343249204) < 1e-12);
        EXPECT(fabs(H[0] - 2.193175735890015) < 1e-12 && fabs(H[1] - 5.284782467867294) < 1e-12);
    }
    /* Random f64 and bf16 problems: every variant, row lists and thread counts agree. */
    enum { T = 7, D = 24, F = 520 }; /* F > 256: column ranges split across tasks */
    double *X = malloc(sizeof(double) * T * D), *Wg = malloc(sizeof(double) * D * F);
    double *Wu = malloc(sizeof(double) * D * F), *Wd = malloc(sizeof(double) * F * D);
    uint16_t *Xb = malloc(2 * T * D), *Wgb = malloc(2 * D * F), *Wub = malloc(2 * D * F), *Wdb = malloc(2 * F * D);
    fill(X, T * D, 1.0), fill(Wg, D * F, 0.2), fill(Wu, D * F, 0.2), fill(Wd, F * D, 0.05);
    fill_bf16(Xb, T * D, 1.0), fill_bf16(Wgb, D * F, 0.2), fill_bf16(Wub, D * F, 0.2), fill_bf16(Wdb, F * D, 0.05);
    const int64_t rows[5] = {6, 0, 3, 3, 1};
    double all[T * D], allH[T * F], part[5 * D], partH[5 * F];
    for (int act = 0; act <= 2; ++act)
        for (int rms = 0; rms <= 1; ++rms)
            for (int threads = 1; threads <= 4; threads += 3) {
                EXPECT(gmlp_oracle_variant_rows_f64(X, Wg, Wu, Wd, T, D, F, act, 1.702, rms, 1e-5, NULL, T, all,
                                                    allH, threads) == 0);
                EXPECT(gmlp_oracle_variant_rows_f64(X, Wg, Wu, Wd, T, D, F, act, 1.702, rms, 1e-5, rows, 5, part,
                                                    partH, 4 - threads + 1) == 0);
                for (int r = 0; r < 5; ++r) {
                    EXPECT(same(part + r * D, all + rows[r] * D, D));
                    EXPECT(same(partH + r * F, allH + rows[r] * F, F));
                }
                EXPECT(gmlp_oracle_variant_rows_bf16(Xb, Wgb, Wub, Wdb, T, D, F, act, 0.5, rms, 0.0, NULL, T, all,
                                                     NULL, threads) == 0);
                EXPECT(gmlp_oracle_variant_rows_bf16(Xb, Wgb, Wub, Wdb, T, D, F, act, 0.5, rms, 0.0, rows, 5, part,
                                                     NULL, threads) == 0);
                for (int r = 0; r < 5; ++r)
                    EXPECT(same(part + r * D, all + rows[r] * D, D));
                for (int i = 0; i < T * D; ++i)
                    EXPECT(isfinite(all[i]));
            }
    /* The down step alone on rows of a bf16 H [T, F]. */
    {
        uint16_t *Hb = malloc(2 * T * F);
        fill_bf16(Hb, T * F, 1.0);
        EXPECT(gmlp_oracle_down_rows_bf16(Hb, Wdb, T, F, D, NULL, T, all, 2) == 0);
        EXPECT(gmlp_oracle_down_rows_bf16(Hb, Wdb, T, F, D, rows, 5, part, 1) == 0);
        for (int r = 0; r < 5; ++r)
            EXPECT(same(part + r * D, all + rows[r] * D, D));
        EXPECT(gmlp_oracle_down_rows_bf16(Hb, Wdb, T, F, D, rows, -1, part, 1) == 1);
        free(Hb);
    }
    /* Errors and empty row lists. */
    const int64_t bad[2] = {0, T};
    EXPECT(gmlp_oracle_rows_f64(X, Wg, Wu, Wd, T, D, F, bad, 2, part, NULL, 1) == 2);
    EXPECT(gmlp_oracle_rows_f64(NULL, Wg, Wu, Wd, T, D, F, NULL, 1, part, NULL, 1) == 1);
    EXPECT(gmlp_oracle_rows_f64(X, Wg, Wu, Wd, T, 0, F, NULL, 1, part, NULL, 1) == 1);
    EXPECT(gmlp_oracle_variant_rows_f64(X, Wg, Wu, Wd, T, D, F, 3, 1.0, 0, 0.0, NULL, 1, part, NULL, 1) == 1);
    EXPECT(gmlp_oracle_variant_rows_f64(X, Wg, Wu, Wd, T, D, F, 0, 1.0, 1, -1.0, NULL, 1, part, NULL, 1) == 1);
    EXPECT(gmlp_oracle_rows_f64(X, Wg, Wu, Wd, T, D, F, NULL, 0, part, NULL, 1) == 0);

    /* Softmax+MatMul: X [M, K] logits, Y [K, N]. */
    enum { M = 6, K = 300, N = 40 };
    double *SX = malloc(sizeof(double) * M * K), *SY = malloc(sizeof(double) * K * N);
    double Z[M * N], A[M * K], Zp[5 * N];
    fill(SX, M * K, 3.0), fill(SY, K * N, 1.0);
    const int64_t srows[5] = {5, 0, 2, 2, 4};
    for (int threads = 1; threads <= 4; threads += 3) {
        EXPECT(smm_oracle_rows_f64(SX, SY, M, K, N, NULL, M, Z, A, threads) == 0);
        EXPECT(smm_oracle_rows_f64(SX, SY, M, K, N, srows, 5, Zp, NULL, threads) == 0);
        for (int r = 0; r < 5; ++r)
            EXPECT(same(Zp + r * N, Z + srows[r] * N, N));
        for (int i = 0; i < M; ++i) {
            double s = 0.0;
            for (int k = 0; k < K; ++k)
                s += A[i * K + k];
            EXPECT(fabs(s - 1.0) < 1e-12);
        }
    }
    uint16_t *SXb = malloc(2 * M * K), *SYb = malloc(2 * K * N);
    fill_bf16(SXb, M * K, 2.0), fill_bf16(SYb, K * N, 1.0);
    EXPECT(smm_oracle_rows_bf16(SXb, SYb, M, K, N, NULL, M, Z, NULL, 2) == 0);
    SX[3 * K + 7] = 1000.0; /* exp overflows double: row 3 is outside the oracle's domain */
    EXPECT(smm_oracle_rows_f64(SX, SY, M, K, N, NULL, M, Z, NULL, 2) == 4);
    EXPECT(smm_oracle_rows_f64(SX, SY, M, K, N, srows, 1, Z, NULL, 2) == 0); /* row 5 only */
    const int64_t sbad[1] = {M};
    EXPECT(smm_oracle_rows_f64(SX, SY, M, K, N, sbad, 1, Z, NULL, 1) == 2);

    free(X), free(Wg), free(Wu), free(Wd), free(Xb), free(Wgb), free(Wub), free(Wdb);
    free(SX), free(SY), free(SXb), free(SYb);
    printf("oracle: %d failures\n", failures);
    return failures ? 1 : 0;
}
