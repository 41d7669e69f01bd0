/*
 * CPU fp64 oracle for Softmax+MatMul:  Z = softmax(X) Y.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or helper
 * with the HIP library.
 *
 * What it computes is the graph of the paper's Fig. "Softmax+MatMul"
 * (fig:softmax-matmul-comp-graph (a), Appendix B), written out for
 * X [M, K] and Y [K, N]:
 *   exp:     E[i, k] = exp(X[i, k])
 *   sum:     S[i]    = sum over k of E[i, k]          (along each row)
 *   divide:  A[i, k] = E[i, k] / S[i]
 *   matmul:  Z[i, j] = sum over k of A[i, k] Y[k, j]   (Fig. fig:op-sema)
 * The softmax runs along the axis the matmul contracts; that is why the
 * divide commutes with the matmul (Appendix B), but the oracle keeps the
 * order of graph (a): normalise first, multiply second.
 *
 * Every step is done in IEEE double precision (the build passes
 * -ffp-contract=off), sums in ascending k order; bf16 inputs are decoded
 * exactly.  exp is taken of X itself, as in the graph, so the oracle's
 * domain is the rows whose exp and sum stay finite and nonzero in double
 * precision (entries below about 709.7, and at least one above about -745);
 * for any other row the entry points return 4 instead of inf or NaN.
 *
 * Rows of X are independent, so the entry points take a list of rows and
 * compute only those (large shapes are checked on sampled rows).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static inline double smm_ld_f64(const double *p, int64_t i) { return p[i]; }
static inline double smm_ld_bf16(const uint16_t *p, int64_t i)
{
    uint32_t u = (uint32_t)p[i] << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Width of the column ranges handed to threads when few rows are requested. */
#define SMM_CHUNK 256

static int smm_threads(int threads)
{
    if (threads > 0)
        return threads;
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * Row steps for one element type WT decoded by LD:
 *
 *   softmax_row: a[k] = exp(x[k]) / sum_k' exp(x[k'])   (returns 4 when the
 *                row is outside the domain described above)
 *   matmul_cols: z[j] = sum_k a[k] Y[k, j] for j in [j_lo, j_hi)
 */
#define DEFINE_SMM_STEPS(SUF, WT, LD)                                           \
    static int softmax_row_##SUF(const WT *X, int64_t t, int64_t K, double *a)  \
    {                                                                           \
        double s = 0.0;                                                         \
        for (int64_t k = 0; k < K; ++k) {                                       \
            a[k] = exp(LD(X, t * K + k));                                       \
            s += a[k];                                                          \
        }                                                                       \
        if (!(s > 0.0) || !isfinite(s))                                         \
            return 4;                                                           \
        for (int64_t k = 0; k < K; ++k)                                         \
            a[k] = a[k] / s;                                                    \
        return 0;                                                               \
    }                                                                           \
    static void matmul_cols_##SUF(const double *a, const WT *Y, int64_t K,      \
                                  int64_t N, int64_t j_lo, int64_t j_hi,        \
                                  double *z)                                    \
    {                                                                           \
        for (int64_t j = j_lo; j < j_hi; ++j)                                   \
            z[j] = 0.0;                                                         \
        for (int64_t k = 0; k < K; ++k) {                                       \
            double ak = a[k];                                                   \
            for (int64_t j = j_lo; j < j_hi; ++j)                               \
                z[j] += ak * LD(Y, k * N + j);                                  \
        }                                                                       \
    }

DEFINE_SMM_STEPS(bf16, uint16_t, smm_ld_bf16)
DEFINE_SMM_STEPS(f64, double, smm_ld_f64)

/*
 * Entry points.  X [M, K] and Y [K, N] are row-major.  rows[n] lists the rows
 * of X to evaluate (NULL means rows 0..n-1).  Outputs: Z [n, N] and, if A is
 * not NULL, A [n, K] (the softmax of those rows).  threads <= 0 uses the
 * OpenMP default.  Returns 0 on success, 1 on a bad argument, 2 on a row
 * index outside [0, M), 3 on allocation failure, 4 on a row outside the
 * oracle's domain.
 */
#define SMM_DRIVER(SUF)                                                         \
    if (K <= 0 || N <= 0 || M < 0 || n < 0 || !X || !Y || !Z)                   \
        return 1;                                                               \
    for (int64_t r = 0; r < n; ++r) {                                           \
        int64_t t = rows ? rows[r] : r;                                         \
        if (t < 0 || t >= M)                                                    \
            return 2;                                                           \
    }                                                                           \
    if (n == 0)                                                                 \
        return 0;                                                               \
    int nthr = smm_threads(threads);                                            \
    double *a_all = (double *)malloc(sizeof(double) * (size_t)n * (size_t)K);   \
    if (!a_all)                                                                 \
        return 3;                                                               \
    int bad = 0;                                                                \
    _Pragma("omp parallel for num_threads(nthr) schedule(dynamic, 1) reduction(|:bad)") \
    for (int64_t r = 0; r < n; ++r)                                             \
        bad |= softmax_row_##SUF(X, rows ? rows[r] : r, K, a_all + r * K);      \
    if (bad) {                                                                  \
        free(a_all);                                                            \
        return 4;                                                               \
    }                                                                           \
    /* Many rows: one row per task.  Few rows: column ranges per task. */       \
    int64_t jc = n >= nthr ? N : SMM_CHUNK;                                     \
    int64_t njc = (N + jc - 1) / jc;                                            \
    _Pragma("omp parallel for num_threads(nthr) schedule(dynamic, 1)")          \
    for (int64_t task = 0; task < n * njc; ++task) {                            \
        int64_t r = task / njc, j_lo = (task % njc) * jc;                       \
        int64_t j_hi = j_lo + jc < N ? j_lo + jc : N;                           \
        matmul_cols_##SUF(a_all + r * K, Y, K, N, j_lo, j_hi, Z + r * N);       \
    }                                                                           \
    if (A)                                                                      \
        memcpy(A, a_all, sizeof(double) * (size_t)n * (size_t)K);               \
    free(a_all);                                                                \
    return 0;

int smm_oracle_rows_bf16(const uint16_t *X, const uint16_t *Y, int64_t M, int64_t K, int64_t N,
                         const int64_t *rows, int64_t n, double *Z, double *A, int threads)
{
    SMM_DRIVER(bf16)
}

int smm_oracle_rows_f64(const double *X, const double *Y, int64_t M, int64_t K, int64_t N,
                        const int64_t *rows, int64_t n, double *Z, double *A, int threads)
{
    SMM_DRIVER(f64)
}
