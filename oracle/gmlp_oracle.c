/*
 * CPU fp64 oracle for the Gated MLP  Y = (act(X Wg) * (X Wu)) Wd  and its
 * variants.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or helper
 * with the HIP library.
 *
 * What it computes is the plain definition, written out:
 *   - the Gated MLP graph of the paper's Fig. "Gated MLP" (fig:mlp-example,
 *     Section 4.2): X feeds two matmuls (W1 -> silu, W2), their results are
 *     multiplied elementwise, and the product feeds a third matmul with W3.
 *     Here W1 = Wg (gate), W2 = Wu (up), W3 = Wd (down).
 *   - matmul(a, b)[i, j] = sum over k of a[i, k] * b[k, j]  (matmul semantics,
 *     Fig. fig:op-sema in Section 4.2.1, and the granular-operation table
 *     tab:nki-ops in Section 5.1).
 *   - silu(x) = x * sigmoid(x)  (granular-operation table tab:nki-ops).
 * Variants (the paper's benchmark list in Section 6.1 names SwiGLU and GLU
 * and a SwiGLU Gated MLP, without formulas; the usual definitions are used):
 *   - swish_beta(g) = g * sigmoid(beta * g)  (the SwiGLU gate; beta = 1 is
 *     silu), and sigmoid(g) (the GLU gate) in place of silu;
 *   - RMSNorm in front (Section 2, the RMSNorm equation): each row x of X is
 *     replaced by x / sqrt(mean(x^2) + eps) before the two matmuls.
 *
 * Every step is done in IEEE double precision (no fused multiply-add: the
 * build passes -ffp-contract=off).  bf16 inputs are decoded exactly (a bf16
 * is the top 16 bits of an IEEE binary32), so the oracle sees exactly the
 * values the GPU sees.  Each output element is accumulated in ascending
 * index order; the loop over output columns is only placed inside the
 * reduction loop for memory order, which leaves every element's own
 * accumulation order unchanged.
 *
 * Rows of X are independent, so the entry points take a list of rows and
 * compute only those (this lets large shapes be checked on sampled rows).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* silu(z) = z * sigmoid(z) = z / (1 + exp(-z)).  For z < 0 the algebraically
 * equal form z * exp(z) / (1 + exp(z)) is used so that exp never overflows. */
double gmlp_oracle_silu(double z)
{
    if (z >= 0.0)
        return z / (1.0 + exp(-z));
    double e = exp(z);
    return z * e / (1.0 + e);
}

/* sigmoid(z) = 1 / (1 + exp(-z)), with exp(z) / (1 + exp(z)) for z < 0 so
 * that exp never overflows. */
double gmlp_oracle_sigmoid(double z)
{
    if (z >= 0.0)
        return 1.0 / (1.0 + exp(-z));
    double e = exp(z);
    return e / (1.0 + e);
}

/* Gate activations (the values of the library's enum gmlp_activation). */
#define ORACLE_ACT_SILU 0
#define ORACLE_ACT_SWISH 1
#define ORACLE_ACT_SIGMOID 2

/* act(g): silu(g), g * sigmoid(beta * g), or sigmoid(g). */
double gmlp_oracle_gate(double g, int act, double beta)
{
    switch (act) {
    case ORACLE_ACT_SILU: return gmlp_oracle_silu(g);
    case ORACLE_ACT_SWISH: return g * gmlp_oracle_sigmoid(beta * g);
    default: return gmlp_oracle_sigmoid(g);
    }
}

/* Exact bf16 -> double: the 16 bits are the high half of a binary32. */
double gmlp_oracle_bf16_to_f64(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static inline double ld_f64(const double *p, int64_t i) { return p[i]; }
static inline double ld_bf16(const uint16_t *p, int64_t i)
{
    uint32_t u = (uint32_t)p[i] << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * The two steps of one row (x already decoded, and normalised if asked),
 * for weights of one element type WT decoded by LD:
 *
 *   gate_up: for f in [f_lo, f_hi):
 *              G[f] = sum_d x[d] Wg[d, f]      (d ascending)
 *              U[f] = sum_d x[d] Wu[d, f]      (d ascending)
 *              H[f] = act(G[f]) * U[f]
 *   down:    for j in [j_lo, j_hi):
 *              Y[j] = sum_f H[f] Wd[f, j]      (f ascending)
 *
 * The column ranges only split work between threads.
 */
#define DEFINE_ROW_STEPS(SUF, WT, LD)                                           \
    static int gate_up_##SUF(const double *x, const WT *Wg, const WT *Wu,       \
                             int64_t D, int64_t F, int64_t f_lo,                \
                             int64_t f_hi, int act, double beta, double *h)     \
    {                                                                           \
        int64_t w = f_hi - f_lo;                                                \
        double *g = (double *)calloc((size_t)w, sizeof(double));                \
        double *u = (double *)calloc((size_t)w, sizeof(double));                \
        if (!g || !u) {                                                         \
            free(g);                                                            \
            free(u);                                                            \
            return 1;                                                           \
        }                                                                       \
        for (int64_t d = 0; d < D; ++d) {                                       \
            double xd = x[d];                                                   \
            for (int64_t j = 0; j < w; ++j) {                                   \
                g[j] += xd * LD(Wg, d * F + f_lo + j);                          \
                u[j] += xd * LD(Wu, d * F + f_lo + j);                          \
            }                                                                   \
        }                                                                       \
        for (int64_t j = 0; j < w; ++j)                                         \
            h[f_lo + j] = gmlp_oracle_gate(g[j], act, beta) * u[j];             \
        free(g);                                                                \
        free(u);                                                                \
        return 0;                                                               \
    }                                                                           \
    static void down_##SUF(const double *h, const WT *Wd, int64_t F,            \
                           int64_t D, int64_t j_lo, int64_t j_hi, double *y)    \
    {                                                                           \
        for (int64_t j = j_lo; j < j_hi; ++j)                                   \
            y[j] = 0.0;                                                         \
        for (int64_t f = 0; f < F; ++f) {                                       \
            double hf = h[f];                                                   \
            for (int64_t j = j_lo; j < j_hi; ++j)                               \
                y[j] += hf * LD(Wd, f * D + j);                                 \
        }                                                                       \
    }

DEFINE_ROW_STEPS(bf16, uint16_t, ld_bf16)
DEFINE_ROW_STEPS(f64, double, ld_f64)

/* Width of the column ranges handed to threads when few rows are requested. */
#define CHUNK 256

static int check_args(const void *X, const void *Wg, const void *Wu, const void *Wd,
                      int64_t T, int64_t D, int64_t F, const int64_t *rows, int64_t n,
                      const double *Y)
{
    if (D <= 0 || F <= 0 || T < 0 || n < 0 || !X || !Wg || !Wu || !Wd || !Y)
        return 1;
    for (int64_t r = 0; r < n; ++r) {
        int64_t t = rows ? rows[r] : r;
        if (t < 0 || t >= T)
            return 2;
    }
    return 0;
}

static int pick_threads(int threads)
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
 * Entry points.  Arrays are row-major: X [T, D], Wg [D, F], Wu [D, F],
 * Wd [F, D].  act selects the gate activation (silu, swish_beta, sigmoid),
 * rms != 0 puts RMSNorm with epsilon eps (>= 0) in front.  rows[n] lists the
 * rows of X to evaluate (NULL means rows 0..n-1).  Outputs: Y [n, D] and, if
 * H is not NULL, H [n, F] (the product act(G) * U before the down
 * projection).  threads <= 0 uses the OpenMP default.  Returns 0 on success,
 * 1 on a bad argument, 2 on a row index outside [0, T), 3 on allocation
 * failure.
 */
#define ORACLE_DRIVER(SUF, WT, LD)                                              \
    int rc = check_args(X, Wg, Wu, Wd, T, D, F, rows, n, Y);                    \
    if (rc)                                                                     \
        return rc;                                                              \
    if (act < ORACLE_ACT_SILU || act > ORACLE_ACT_SIGMOID || (rms && !(eps >= 0.0))) \
        return 1;                                                               \
    if (n == 0)                                                                 \
        return 0;                                                               \
    int nthr = pick_threads(threads);                                           \
    double *h_all = (double *)malloc(sizeof(double) * (size_t)n * (size_t)F);   \
    double *x_all = (double *)malloc(sizeof(double) * (size_t)n * (size_t)D);   \
    if (!h_all || !x_all) {                                                     \
        free(h_all);                                                            \
        free(x_all);                                                            \
        return 3;                                                               \
    }                                                                           \
    /* The rows of X, decoded; with RMSNorm, x[d] * 1/sqrt(mean(x^2) + eps). */ \
    for (int64_t r = 0; r < n; ++r) {                                           \
        int64_t t = rows ? rows[r] : r;                                         \
        double *xr = x_all + r * D;                                             \
        for (int64_t d = 0; d < D; ++d)                                         \
            xr[d] = LD(X, t * D + d);                                           \
        if (rms) {                                                              \
            double ss = 0.0;                                                    \
            for (int64_t d = 0; d < D; ++d)                                     \
                ss += xr[d] * xr[d];                                            \
            double inv = 1.0 / sqrt(ss / (double)D + eps);                      \
            for (int64_t d = 0; d < D; ++d)                                     \
                xr[d] = xr[d] * inv;                                            \
        }                                                                       \
    }                                                                           \
    /* Many rows: one row per task.  Few rows: column ranges per task. */       \
    int64_t fc = n >= nthr ? F : CHUNK, dc = n >= nthr ? D : CHUNK;             \
    int64_t nfc = (F + fc - 1) / fc, ndc = (D + dc - 1) / dc;                   \
    int fail = 0;                                                               \
    _Pragma("omp parallel for num_threads(nthr) schedule(dynamic, 1) reduction(|:fail)") \
    for (int64_t task = 0; task < n * nfc; ++task) {                            \
        int64_t r = task / nfc, f_lo = (task % nfc) * fc;                       \
        int64_t f_hi = f_lo + fc < F ? f_lo + fc : F;                           \
        fail |= gate_up_##SUF(x_all + r * D, Wg, Wu, D, F, f_lo, f_hi, act, beta, \
                              h_all + r * F);                                   \
    }                                                                           \
    free(x_all);                                                                \
    if (fail) {                                                                 \
        free(h_all);                                                            \
        return 3;                                                               \
    }                                                                           \
    _Pragma("omp parallel for num_threads(nthr) schedule(dynamic, 1)")          \
    for (int64_t task = 0; task < n * ndc; ++task) {                            \
        int64_t r = task / ndc, j_lo = (task % ndc) * dc;                       \
        int64_t j_hi = j_lo + dc < D ? j_lo + dc : D;                           \
        down_##SUF(h_all + r * F, Wd, F, D, j_lo, j_hi, Y + r * D);             \
    }                                                                           \
    if (H)                                                                      \
        memcpy(H, h_all, sizeof(double) * (size_t)n * (size_t)F);               \
    free(h_all);                                                                \
    return 0;

int gmlp_oracle_variant_rows_bf16(const uint16_t *X, const uint16_t *Wg, const uint16_t *Wu,
                                  const uint16_t *Wd, int64_t T, int64_t D, int64_t F, int act,
                                  double beta, int rms, double eps, const int64_t *rows, int64_t n,
                                  double *Y, double *H, int threads)
{
    ORACLE_DRIVER(bf16, uint16_t, ld_bf16)
}

int gmlp_oracle_variant_rows_f64(const double *X, const double *Wg, const double *Wu,
                                 const double *Wd, int64_t T, int64_t D, int64_t F, int act,
                                 double beta, int rms, double eps, const int64_t *rows, int64_t n,
                                 double *Y, double *H, int threads)
{
    ORACLE_DRIVER(f64, double, ld_f64)
}

/* The SiLU Gated MLP (no RMSNorm): the variant entry points with act = silu. */
int gmlp_oracle_rows_bf16(const uint16_t *X, const uint16_t *Wg, const uint16_t *Wu,
                          const uint16_t *Wd, int64_t T, int64_t D, int64_t F,
                          const int64_t *rows, int64_t n, double *Y, double *H,
                          int threads)
{
    return gmlp_oracle_variant_rows_bf16(X, Wg, Wu, Wd, T, D, F, ORACLE_ACT_SILU, 1.0, 0, 0.0,
                                         rows, n, Y, H, threads);
}

int gmlp_oracle_rows_f64(const double *X, const double *Wg, const double *Wu,
                         const double *Wd, int64_t T, int64_t D, int64_t F,
                         const int64_t *rows, int64_t n, double *Y, double *H,
                         int threads)
{
    return gmlp_oracle_variant_rows_f64(X, Wg, Wu, Wd, T, D, F, ORACLE_ACT_SILU, 1.0, 0, 0.0,
                                        rows, n, Y, H, threads);
}

/*
 * Step 4 alone, on given rows of a bf16 H [T, F]: Y[r, :] = H[rows[r], :] Wd
 * with Wd [F, D] (the down projection of the graph, checked by itself).
 * Same return codes as above.
 */
int gmlp_oracle_down_rows_bf16(const uint16_t *H, const uint16_t *Wd, int64_t T, int64_t F,
                               int64_t D, const int64_t *rows, int64_t n, double *Y,
                               int threads)
{
    if (D <= 0 || F <= 0 || T < 0 || n < 0 || !H || !Wd || !Y)
        return 1;
    for (int64_t r = 0; r < n; ++r) {
        int64_t t = rows ? rows[r] : r;
        if (t < 0 || t >= T)
            return 2;
    }
    int nthr = pick_threads(threads);
    double *h = (double *)malloc(sizeof(double) * (size_t)n * (size_t)F);
    if (!h)
        return 3;
    for (int64_t r = 0; r < n; ++r) {
        int64_t t = rows ? rows[r] : r;
        for (int64_t f = 0; f < F; ++f)
            h[r * F + f] = ld_bf16(H, t * F + f);
    }
    int64_t dc = n >= nthr ? D : CHUNK;
    int64_t ndc = (D + dc - 1) / dc;
#pragma omp parallel for num_threads(nthr) schedule(dynamic, 1)
    for (int64_t task = 0; task < n * ndc; ++task) {
        int64_t r = task / ndc, j_lo = (task % ndc) * dc;
        int64_t j_hi = j_lo + dc < D ? j_lo + dc : D;
        down_bf16(h + r * F, Wd, F, D, j_lo, j_hi, Y + r * D);
    }
    free(h);
    return 0;
}

/* Number of threads the OpenMP runtime uses by default. */
int gmlp_oracle_max_threads(void)
{
    return pick_threads(0);
}
