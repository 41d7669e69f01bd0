// Row scales of RMSNorm for the MFMA path of the RMSNorm-fused Gated MLP.
//
// RMSNorm (the equation of Section 2) multiplies each row x of X by
// r = 1 / sqrt(mean(x^2) + eps).  The paper's headline reorder moves that
// multiply past the matmul, (x * r) W = r * (x W), so the two parts become
// independent: this kernel computes r for every row while X itself goes to
// the gate/up GEMM unnormalised, and the GEMM epilogue scales G and U by r.
// (The GEMV path computes r inside its gate/up kernel instead.)
#pragma once

#include "common.hpp"

namespace gmlp {

constexpr int kRowRmsThreads = 256; // 4 waves, one row each

// r[t] = 1 / sqrt(sum_d X[t, d]^2 / D + eps), X [T, D] bf16, D a multiple of
// 8.  Each lane adds its 8-element slices in order, then a butterfly over
// the wave (every lane ends with the same, order-fixed sum).
__global__ __launch_bounds__(kRowRmsThreads) void row_rms_kernel(const uint16_t *X, float *r, int T, int D,
                                                                 float eps)
{
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int t = blockIdx.x * (kRowRmsThreads / 64) + wave;
    if (t >= T)
        return;
    const uint16_t *x = X + (size_t)t * D;
    float s = 0.0f;
    for (int d = lane * 8; d < D; d += 64 * 8) {
        const u32x4 v = *(const u32x4 *)(x + d);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float lo = bf16_lo(v[e]), hi = bf16_hi(v[e]);
            s += lo * lo;
            s += hi * hi;
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        s += __shfl_xor(s, off);
    if (lane == 0)
        r[t] = 1.0f / __builtin_sqrtf(s / (float)D + eps);
}

} // namespace gmlp
