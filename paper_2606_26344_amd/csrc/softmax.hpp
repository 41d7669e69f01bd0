// Softmax+MatMul, first part: the exponentials and the row sums.
//
// Z = softmax(X) Y with the softmax along the axis the matmul contracts
// (Appendix B, Fig. fig:softmax-matmul-comp-graph).  Because the softmax's
// normalising sum runs over that same axis, the divide commutes with the
// matmul: (E / s) Y = (E Y) / s row by row.  So this kernel writes the
// unnormalised exponentials and their row sums, the matmul consumes the
// exponentials directly, and the divide happens in the GEMM's epilogue on
// the [M, N] result instead of on the [M, K] operand.
//
// Per row i of X [M, K] (bf16, K a multiple of 8):
//   m_i     = max_k X[i, k]
//   P[i, k] = bf16(exp(X[i, k] - m_i))                 (round to nearest even)
//   s[i]    = sum_k exp(X[i, k] - m_i)                  (fp32, unrounded terms)
// Subtracting m_i leaves the softmax unchanged (exp(x - m) / sum exp(x - m)
// = exp(x) / sum exp(x)), keeps every exponential in (0, 1] and makes
// 1 <= s[i] <= K.  A row holding NaN, +inf, or only -inf yields NaN.
#pragma once

#include "common.hpp"

namespace gmlp {

constexpr int kSoftmaxThreads = 256; // 4 waves, one row each
// 16-byte chunks (8 columns) per lane held in registers: rows of up to
// 64 * 16 * 8 = 8192 columns are read from memory once; longer rows are read
// twice (a max pass, then the exponentials), the second time mostly from cache.
constexpr int kSoftmaxMaxChunks = 16;

// Butterfly reductions over the 64 lanes: every lane ends with the same
// value, combined in the same fixed order on every run.
__device__ __forceinline__ float wave_max(float v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        v = fmaxf(v, __shfl_xor(v, off));
    return v;
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        v += __shfl_xor(v, off);
    return v;
}

// R chunks of one lane, starting at chunk c0 + lane.  Chunks past the row
// end re-read the last chunk (an unconditional, in-bounds load); callers
// mask them where it matters.
template <int R>
__device__ __forceinline__ void load_chunks(const uint16_t *x, int c0, int lane, int nchunk, u32x4 (&v)[R])
{
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int c = c0 + lane + 64 * r;
        v[r] = *(const u32x4 *)(x + 8 * (c < nchunk ? c : nchunk - 1));
    }
}

// A repeated chunk cannot change a maximum, so no mask is needed.
template <int R>
__device__ __forceinline__ float chunks_max(const u32x4 (&v)[R], float m)
{
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int e = 0; e < 4; ++e)
            m = fmaxf(m, fmaxf(bf16_lo(v[r][e]), bf16_hi(v[r][e])));
    return m;
}

// exp(x - m) of the lane's valid chunks: stored as bf16, added to `sum` in
// column order.
template <int R>
__device__ __forceinline__ float chunks_exp(const u32x4 (&v)[R], uint16_t *p, int c0, int lane, int nchunk,
                                            float m, float sum)
{
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int c = c0 + lane + 64 * r;
        if (c < nchunk) {
            u32x4 out;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float lo = __expf(bf16_lo(v[r][e]) - m);
                const float hi = __expf(bf16_hi(v[r][e]) - m);
                sum += lo;
                sum += hi;
                out[e] = pack_bf16x2(lo, hi);
            }
            *(u32x4 *)(p + 8 * c) = out;
        }
    }
    return sum;
}

// One wave per row.  R (<= kSoftmaxMaxChunks) chunks per lane cover the row
// when K <= 512 R; otherwise the row is streamed in pieces of 512 R columns.
// The per-lane sums run over the lane's chunks in ascending column order in
// both cases, so s does not depend on which case ran.
template <int R>
__global__ __launch_bounds__(kSoftmaxThreads) void softmax_exp_rows_kernel(const uint16_t *X, uint16_t *P,
                                                                           float *s, int M, int K)
{
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int i = blockIdx.x * (kSoftmaxThreads / 64) + wave;
    if (i >= M)
        return;
    const uint16_t *x = X + (size_t)i * K;
    uint16_t *p = P + (size_t)i * K;
    const int nchunk = K >> 3;
    u32x4 v[R];
    float m = -__builtin_inff(), sum = 0.0f;
    if (nchunk <= 64 * R) {
        load_chunks<R>(x, 0, lane, nchunk, v);
        m = wave_max(chunks_max<R>(v, m));
        sum = chunks_exp<R>(v, p, 0, lane, nchunk, m, sum);
    } else {
        for (int c0 = 0; c0 < nchunk; c0 += 64 * R) {
            load_chunks<R>(x, c0, lane, nchunk, v);
            m = chunks_max<R>(v, m);
        }
        m = wave_max(m);
        for (int c0 = 0; c0 < nchunk; c0 += 64 * R) {
            load_chunks<R>(x, c0, lane, nchunk, v);
            sum = chunks_exp<R>(v, p, c0, lane, nchunk, m, sum);
        }
    }
    sum = wave_sum(sum);
    if (lane == 0)
        s[i] = sum;
}

// Chunks per lane for a row of K columns: the smallest power of two that
// holds the row, at most kSoftmaxMaxChunks.
inline int softmax_chunks_per_lane(int K)
{
    const int nchunk = K / 8;
    int r = 1;
    while (r < kSoftmaxMaxChunks && 64 * r < nchunk)
        r *= 2;
    return r;
}

} // namespace gmlp
