/*
 * softmax_matmul.h -- C ABI of the MI355X (gfx950) Softmax+MatMul kernels in
 * libgmlp.so.
 *
 * The operation (the paper's "Softmax+MatMul" benchmark; graph in Fig.
 * fig:softmax-matmul-comp-graph, Appendix B):
 *
 *     Z = softmax(X) Y,   softmax(x)[k] = exp(x[k]) / sum_k' exp(x[k'])
 *
 * with the softmax taken along each row of X, which is the axis the matmul
 * contracts.  The normalising sum therefore reduces along the contracted
 * axis and the divide commutes with the matmul (Appendix B):
 * (E / s) Y = (E Y) / s row by row, E = exp(X).  The library computes it in
 * that reordered form: one kernel writes P = exp(X - m) (m the row maximum,
 * which cancels in the quotient) and the row sums s, the matmul consumes P,
 * and the divide by s happens on the [M, N] result in the matmul's epilogue.
 *
 * Numerics: X, Y and Z are IEEE bfloat16 (bit patterns in uint16 storage).
 * exp(x - m) and s are computed in fp32; P is rounded once to bf16
 * (round-to-nearest-even) and s sums the unrounded fp32 exponentials;
 * products are accumulated in fp32 and divided by s in fp32 (IEEE division);
 * Z is rounded once to bf16.  A row of X holding NaN or +inf, or only -inf,
 * gives a NaN row of Z.
 *
 * Layout: dense, row-major, on the current HIP device:
 *     X [M, K]     Y [K, N]     Z [M, N]
 * K and N must be multiples of 8 (at most 2^22), M at most 2^24, no tensor
 * may hold more than 2^37 elements, and every pointer must be 16-byte
 * aligned.  M == 0 is valid and launches nothing.
 *
 * Ownership, streams and errors are as in gmlp.h: the caller owns every
 * buffer; calls only enqueue work on `stream` (a hipStream_t, NULL = null
 * stream); every entry point returns GMLP_OK or a positive GMLP_ERR_* code
 * (enum gmlp_status) with a detail in gmlp_last_error().
 */
#ifndef SOFTMAX_MATMUL_H
#define SOFTMAX_MATMUL_H

#include <stddef.h>
#include <stdint.h>

#include "gmlp.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Bytes of workspace softmax_matmul_ws needs for this shape (any path): the
 * exponentials P [M, K] bf16, the row sums [M] fp32, fp32 split-K partial
 * sums of the matmul and the block of arrival counters that
 * gmlp_workspace_init zeroes.  0 if the shape is invalid.
 */
size_t softmax_matmul_workspace_size(int64_t M, int64_t K, int64_t N);

/*
 * The kernels softmax_matmul_ws(..., path, ...) enqueues for this shape, in
 * the format of gmlp_describe: first the exponential/row-sum kernel, then
 * the matmul (path as in enum gmlp_path: GEMV for M <= 8 under
 * GMLP_PATH_AUTO, MFMA GEMM otherwise).  Host-only.  Nothing for M == 0.
 */
int softmax_matmul_describe(int64_t M, int64_t K, int64_t N, int path, char *buf, size_t bytes);

/*
 * Z = softmax(X) Y for X [M, K], Y [K, N], Z [M, N] bf16 device pointers,
 * with a caller workspace of `ws_bytes` >= softmax_matmul_workspace_size
 * bytes, 256-byte aligned, prepared once with gmlp_workspace_init.  Allocates
 * nothing; enqueues exactly two kernels.  INVALID_ARG for a NULL pointer, a
 * negative size or Z overlapping X, Y or the workspace; UNSUPPORTED for K or
 * N not a multiple of 8, a misaligned pointer or a size beyond the limits;
 * NO_MEMORY for a workspace that is too small.
 */
int softmax_matmul_ws(const void *X, const void *Y, void *Z, int64_t M, int64_t K, int64_t N,
                      int path, void *workspace, size_t ws_bytes, void *stream);

/* softmax_matmul_ws with scratch allocated stream-ordered on `stream` and the
 * automatic path. */
int softmax_matmul(const void *X, const void *Y, void *Z, int64_t M, int64_t K, int64_t N,
                   void *stream);

/*
 * The two halves of the reordered graph (Fig. fig:softmax-matmul-comp-graph
 * (b)), each one kernel; softmax_matmul_ws is exactly the first followed by
 * the second on its workspace's P and s, bit for bit.
 *
 * softmax_matmul_exp_rows: the exp and the row sum.  For X [M, K] bf16,
 * writes P [M, K] bf16 with P[i, k] = bf16(exp(X[i, k] - m_i)), m_i the row
 * maximum, and s [M] fp32 with s[i] = sum_k exp(X[i, k] - m_i) (of the
 * unrounded exponentials).  X, P: 16-byte aligned; s: 4-byte aligned; P and
 * s must not overlap X or each other.  Allocates nothing.
 */
int softmax_matmul_exp_rows(const void *X, void *P, float *s, int64_t M, int64_t K, void *stream);

/*
 * softmax_matmul_divide_ws: the matmul and then the divide,
 * Z[i, :] = bf16((P[i, :] Y) / s[i]) with fp32 accumulation and IEEE fp32
 * division, for P [M, K] bf16, s [M] fp32 (any finite or non-finite values;
 * the caller's), Y [K, N] bf16, Z [M, N] bf16.  Workspace and path as for
 * softmax_matmul_ws (its P and s regions are not used).  Allocates nothing.
 */
int softmax_matmul_divide_ws(const void *P, const float *s, const void *Y, void *Z, int64_t M,
                             int64_t K, int64_t N, int path, void *workspace, size_t ws_bytes,
                             void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SOFTMAX_MATMUL_H */
