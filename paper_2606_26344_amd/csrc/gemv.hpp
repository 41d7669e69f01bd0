// Split-K streaming GEMV kernels of the Gated MLP for few tokens (T <= 8).
//
// With T <= 8 every weight byte is used for at most 8 multiply-adds, so the
// matmuls of the Gated MLP (Fig. fig:mlp-example, Section 4.1) are bound by
// the rate at which the weights stream from HBM.  Each block streams a strip
// of up to 256 weight columns over a slice of k rows:
//
//   * lane (l % 32) owns 8 adjacent columns (one 16-byte load per row); the
//     two 32-lane halves of a wave and the 4 waves take rows k = g, g+8, ...
//     (8 row groups), so a wave reads two 512-byte row segments per load
//     instruction;
//   * the activations of the slice are staged once in LDS as fp32;
//   * partial sums are reduced in a fixed order: across the two halves of
//     the wave by a lane shuffle, across the 4 waves through LDS, and across
//     the split-K blocks of a strip by the last block to finish (arrival
//     counter), which adds the per-block sums in split order;
//   * each lane keeps two batches of 16-byte weight loads in flight (the
//     next batch is issued before the current one is consumed).
//   The result is therefore bitwise reproducible run to run.
//
// The gate/up instantiation (NW = 2) streams Wg and Wu together and its last
// block applies H = bf16(silu(G) * U); the down instantiation (NW = 1)
// streams Wd and writes Y = bf16(H Wd).
#pragma once

#include "common.hpp"

namespace gmlp {

struct GemvParams {
    const uint16_t *w0;  // [K, M] bf16 (Wg, or Wd)
    const uint16_t *w1;  // [K, M] bf16 (Wu) for the gate/up kernel
    const uint16_t *act; // [NT, K] bf16 (X, or H)
    uint16_t *out;       // [NT, M] bf16 (H, or Y)
    float *partial;      // [splits][NW][NT][M] fp32 per-block sums
    uint32_t *counters;  // arrival counter per strip (zero on entry and exit)
    int M, K;
    int k_split;     // rows per split, <= gemv_max_split_rows<NT>()
    int splits;
    int strips;
    int strip_lanes; // lanes per row (8 columns each, <= 32): strip width 8 * strip_lanes
};

constexpr int kGemvMaxStrip = 256; // widest strip (32 lanes x 8 columns)
constexpr int kGemvThreads = 256;

// Weight rows per lane per load batch: 2*NW*U loads of 16 bytes in flight
// per lane (two batches), within the register budget of NT tokens.
template <int NT, int NW>
constexpr int gemv_batch_rows() { return NT <= 2 ? (NW == 1 ? 16 : 8) : 4; }

// Rows of one split: the split's activations are staged in LDS as fp32
// (NT x rows floats, at most 16 KB).
template <int NT>
constexpr int gemv_max_split_rows() { return NT <= 2 ? 2048 : 4096 / NT; }

template <int NT, int NW, int EPI>
__global__ __launch_bounds__(kGemvThreads) void gemv_splitk_kernel(GemvParams p)
{
    constexpr int RG = 8; // row groups per block
    constexpr int U = gemv_batch_rows<NT, NW>();
    __shared__ float xs[NT][gemv_max_split_rows<NT>()];
    __shared__ float red[4][NW][NT][kGemvMaxStrip];
    __shared__ int s_last;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int strip = blockIdx.x % p.strips;
    const int split = blockIdx.x / p.strips;
    const int M = p.M, K = p.K;
    const int width = 8 * p.strip_lanes;
    const int m0 = strip * width;
    const int kb = split * p.k_split;
    const int nrows = min(K, kb + p.k_split) - kb;

    const int col = (lane & 31) * 8;
    const int rg = wave * 2 + (lane >> 5);
    const bool valid = (lane & 31) < p.strip_lanes && m0 + col < M;

    // Weight rows of batch b: rg + 8*(b*U + u), u < U; every lane of the
    // block runs the same nb batches, the last of which may be partial
    // (rows past the split are neither loaded nor accumulated).  The loads
    // bypass caching (each weight byte is read once).
    const uint16_t *wp[NW];
    wp[0] = p.w0 + (size_t)kb * M + m0 + col;
    if constexpr (NW == 2)
        wp[1] = p.w1 + (size_t)kb * M + m0 + col;
    auto load_batch = [&](u32x4 (&v)[U][NW], int b) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = rg + RG * (b * U + u);
#pragma unroll
            for (int w = 0; w < NW; ++w)
                v[u][w] = r < nrows ? __builtin_nontemporal_load((const u32x4 *)(wp[w] + (size_t)r * M))
                                    : u32x4{0u, 0u, 0u, 0u};
        }
    };
    const int nb = (nrows + RG * U - 1) / (RG * U);
    u32x4 va[U][NW], vb[U][NW];
    // The first weight batch is in flight while the activations are staged.
    if (valid && nb > 0)
        load_batch(va, 0);

    // Stage this slice of the activations as fp32.
    for (int i = tid; i < NT * nrows; i += kGemvThreads) {
        const int t = i / nrows, r = i - t * nrows;
        xs[t][r] = __builtin_bit_cast(float, (uint32_t)p.act[(size_t)t * K + kb + r] << 16);
    }
    __syncthreads();

    float acc[NW][NT][8];
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int e = 0; e < 8; ++e)
                acc[w][t][e] = 0.0f;

    if (valid) {
        auto fma_row = [&](const u32x4 (&v)[NW], int r) __attribute__((always_inline)) {
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const float x = xs[t][r];
#pragma unroll
                for (int w = 0; w < NW; ++w)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        acc[w][t][2 * e] += x * bf16_lo(v[w][e]);
                        acc[w][t][2 * e + 1] += x * bf16_hi(v[w][e]);
                    }
            }
        };
        auto fma_batch = [&](const u32x4 (&v)[U][NW], int b) __attribute__((always_inline)) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int r = rg + RG * (b * U + u);
                if (r < nrows)
                    fma_row(v[u], r);
            }
        };
        for (int b = 0; b < nb; b += 2) {
            if (b + 1 < nb)
                load_batch(vb, b + 1);
            fma_batch(va, b);
            if (b + 2 < nb)
                load_batch(va, b + 2);
            if (b + 1 < nb)
                fma_batch(vb, b + 1);
        }
    }

    // Row groups 2*wave and 2*wave+1 share columns: add the two wave halves.
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int e = 0; e < 8; ++e)
                acc[w][t][e] += __shfl_xor(acc[w][t][e], 32);
    if (lane < 32) {
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                f32x4 lo = {acc[w][t][0], acc[w][t][1], acc[w][t][2], acc[w][t][3]};
                f32x4 hi = {acc[w][t][4], acc[w][t][5], acc[w][t][6], acc[w][t][7]};
                *(f32x4 *)&red[wave][w][t][col] = lo;
                *(f32x4 *)&red[wave][w][t][col + 4] = hi;
            }
    }
    __syncthreads();

    // Thread tid now owns column m0 + tid of the strip.
    const int m = m0 + tid;
    const bool mvalid = tid < width && m < M;
    float v[NW][NT];
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int t = 0; t < NT; ++t)
            v[w][t] = ((red[0][w][t][tid] + red[1][w][t][tid]) + red[2][w][t][tid]) + red[3][w][t][tid];

    if (p.splits > 1) {
        // Per-block sums go out with device-coherent stores; once they have
        // completed (vmcnt 0) the block counts itself in.  The block that
        // arrives last reads every split's sums with device-coherent loads.
        // No cache-wide write-back or invalidate is needed.
        if (mvalid) {
#pragma unroll
            for (int w = 0; w < NW; ++w)
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    __hip_atomic_store(&p.partial[(((size_t)split * NW + w) * NT + t) * M + m], v[w][t],
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        wait_vmcnt<0>();
        __syncthreads();
        if (tid == 0) {
            const uint32_t before =
                __hip_atomic_fetch_add(p.counters + strip, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_last = before == (uint32_t)(p.splits - 1);
        }
        __syncthreads();
        if (!s_last)
            return;
        if (tid == 0)
            __hip_atomic_store(p.counters + strip, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (mvalid) {
            // Sum the splits in order 0, 1, 2, ...; loads are issued eight
            // at a time so their latencies overlap.
            constexpr int B = 8;
#pragma unroll
            for (int w = 0; w < NW; ++w)
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const float own = v[w][t];
                    const float *src = &p.partial[((size_t)w * NT + t) * M + m];
                    const size_t stride = (size_t)NW * NT * M;
                    float s = 0.0f;
                    for (int s0 = 0; s0 < p.splits; s0 += B) {
                        float x[B];
#pragma unroll
                        for (int u = 0; u < B; ++u) {
                            const int sp = s0 + u;
                            x[u] = sp == split ? own
                                   : sp < p.splits
                                       ? __hip_atomic_load(src + sp * stride, __ATOMIC_RELAXED,
                                                           __HIP_MEMORY_SCOPE_AGENT)
                                       : 0.0f;
                        }
#pragma unroll
                        for (int u = 0; u < B; ++u)
                            if (s0 + u < p.splits)
                                s = s0 + u == 0 ? x[u] : s + x[u];
                    }
                    v[w][t] = s;
                }
        }
    }

    if (mvalid) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            float y;
            if constexpr (EPI == EPI_SILU_MUL)
                y = silu(v[0][t]) * v[NW - 1][t];
            else
                y = v[0][t];
            p.out[(size_t)t * M + m] = __builtin_bit_cast(uint16_t, (__bf16)y);
        }
    }
}

} // namespace gmlp
