// Split-K streaming GEMV kernels of the Gated MLP for few tokens (T <= 8).
//
// With T <= 8 every weight byte is used for at most 8 multiply-adds, so the
// matmuls of the Gated MLP (Fig. fig:mlp-example, Section 4.2) are bound by
// the rate at which the weights stream from HBM.  A work item streams a strip
// of up to 256 weight columns over a slice of k rows:
//
//   * a lane owns 8 adjacent columns (one 16-byte load per row), and the
//     block's row groups g = 0 .. RG-1 take rows in turn (GemvLayout): a row
//     group is a wave reading one 1 KB row segment per load instruction
//     (gate/up up to 4 tokens: 512-column strips) or a 32-lane half-wave
//     reading 512 bytes (256-column strips);
//   * the activations of a lane's rows are loaded into registers with its
//     weights (no LDS staging, so no barrier stalls the first loads);
//   * partial sums are reduced in a fixed order: across the two halves of
//     a wave by a lane shuffle (half-wave row groups), across the waves
//     through LDS in wave order, and across
//     the split-K items of a strip by the last block to finish (arrival
//     counter), which adds the per-item sums in split order;
//   * each lane keeps two batches of 16-byte weight loads in flight (a
//     batch is reissued as soon as it has been consumed).
//   The result is therefore bitwise reproducible run to run.
//
// The gate/up kernel (NW = 2) streams Wg and Wu together and its last block
// applies H = bf16(act(G) * U) (act = silu, swish_beta or sigmoid; with
// RMSNorm, G and U are first scaled by the row's r); the down kernel (NW = 1)
// streams Wd and writes Y = bf16(H Wd).  gemv_fused_kernel (end of file)
// runs the items of both in one launch.
#pragma once

#include "common.hpp"
#include "tiling.hpp"

namespace gmlp {

struct GemvParams {
    const uint16_t *w0;  // [K, M] bf16 (Wg, or Wd)
    const uint16_t *w1;  // [K, M] bf16 (Wu) for the gate/up kernel
    const uint16_t *act; // [NT, K] bf16 (X, or H)
    uint16_t *out;       // [NT, M] bf16 (H, or Y)
    float *partial;      // [splits][NW][NT][M] fp32 per-item sums
    uint32_t *counters;  // arrival counter per strip (zero on entry and exit)
    int counter_stride;  // words between two strips' counters
    int M, K;
    int k_split;     // rows per split (a multiple of the load batch span)
    int splits;
    int strips;
    int strip_lanes; // lanes per row segment (8 columns each): strip width 8 * strip_lanes
    // Gate/up epilogue: activation (enum Activation) and swish slope.
    int activation;
    float beta;
    // RMSNorm (gate/up kernel with RMS = true): eps, and per-split sums of
    // squares of the activations [strips][splits][NT] fp32 when splits > 1.
    float eps;
    float *ssq;
    // Store kernel: per-token divisors [NT] (nullptr: none), the softmax sums
    // of Softmax+MatMul.
    const float *rowdiv;
};

// Splits whose partial sums the last block of a strip loads at once: up to
// 64 values per thread in flight (NT * NW per split; the streaming
// registers are free by then), so few round trips (measured: T = 5..8 steps
// 3-4% faster than with 16 values).
template <int NT, int NW>
constexpr int gemv_reduce_batch() { return NT * NW <= 4 ? 16 : 64 / (NT * NW); }



// LDS of one block: per-wave column sums, per-wave sums of squares of the
// activations (RMSNorm), last-block flag.
template <int NT, int NW>
struct GemvShared {
    float red[GemvLayout<NT, NW>::WAVES][NW][NT][GemvLayout<NT, NW>::STRIP];
    float ssq[GemvLayout<NT, NW>::WAVES][NT];
    int last;
};

// One work item (strip, split) of a GEMV step, run by the whole block.
// RMS (gate/up only): the activations are RMSNorm-ed rows.  By the paper's
// reorder of the RMSNorm multiply past the matmul (Section 2), the block
// streams the raw rows, adds up the squares of the activations it loads
// anyway, and the last block of the strip scales G and U by
// r = 1 / sqrt(sum(x^2) / K + eps) before the activation.
struct NoWait {
    __device__ bool operator()() const { return true; }
};

// One work item (a strip of columns times one split of rows).  Returns
// whether this block wrote the strip's results (the only, or the last, split
// of the strip).  CO writes the results with device-coherent stores and CX
// reads the activations with device-coherent loads (the fused kernel hands H
// from its gate/up blocks to its down blocks through them); with CX the
// weights of the first batches are issued before wait() and the activations
// only after it.  wait() returns whether the activations are ready; if not
// (a bounded wait that gave up), the block's sums are replaced by NaN, so
// every output its strip produces is NaN rather than a wrong number.
template <int NT, int NW, int EPI, bool RMS, bool CO = false, bool CX = false, class Wait = NoWait>
__device__ __forceinline__ bool gemv_item(const GemvParams &p, int item, GemvShared<NT, NW> &sh,
                                          const Wait &wait = Wait{})
{
    static_assert(!RMS || EPI == EPI_GATE_MUL, "RMSNorm belongs to the gate/up step");
    using L = GemvLayout<NT, NW>;
    constexpr int RG = L::RG; // row groups per block
    constexpr int U = gemv_batch_rows<NT, NW>();
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int strip = item % p.strips;
    const int split = item / p.strips;
    const int M = p.M, K = p.K;
    const int width = 8 * p.strip_lanes;
    const int m0 = strip * width;
    const int kb = split * p.k_split;
    const int nrows = min(K, kb + p.k_split) - kb;

    const int col = (tid % L::LANES) * 8;
    const int rg = tid / L::LANES;

    // Batch b covers rows [RG*U*b, RG*U*(b+1)) of the split; row group rg
    // takes the U consecutive rows from (RG*b + rg)*U.  Every lane of the block runs
    // the same nb batches, the last of which may be partial.  A batch is one
    // load of the U activations of each token (issued first) and U weight
    // loads per weight, all unconditional, so the compiler counts them and
    // waits for exactly the batch it consumes: a lane past the strip's last
    // column reloads that column, and a row past the split reloads a row of
    // the split (neither is accumulated into a stored result).  The weight
    // loads bypass caching (each weight byte is read once).
    const int lcol = min(m0 + col, M - 8);
    const uint16_t *wp[NW];
    wp[0] = p.w0 + (size_t)kb * M + lcol;
    if constexpr (NW == 2)
        wp[1] = p.w1 + (size_t)kb * M + lcol;
    const uint16_t *xp = p.act + kb;
    const __amdgpu_buffer_rsrc_t rxp = make_rsrc(xp); // CX: byte offsets stay below 2^27
    constexpr int XW = U / 2; // activation words (2 bf16 each) per token per batch
    struct Batch {
        uint32_t x[NT][XW];
        u32x4 w[U][NW];
    };
    auto load_x = [&](Batch &v, int b) __attribute__((always_inline)) {
        const int r0 = (RG * b + rg) * U;
        // Activation pieces of min(U, 8) rows lie wholly in or out of the
        // split (nrows is a multiple of 8, r0 of U).
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            if constexpr (U >= 8) {
#pragma unroll
                for (int q = 0; q < U / 8; ++q) {
                    const int r = r0 + 8 * q < nrows ? r0 + 8 * q : 0;
                    u32x4 x4;
                    if constexpr (CX)
                        x4 = __builtin_amdgcn_raw_buffer_load_b128(rxp, (uint32_t)(t * K + r) * 2u, 0, kCoherent);
                    else
                        x4 = *(const u32x4 *)(xp + (size_t)t * K + r);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        v.x[t][4 * q + e] = x4[e];
                }
            } else if constexpr (U == 4) {
                const int r = r0 < nrows ? r0 : 0;
                u32x2 x2;
                if constexpr (CX)
                    x2 = __builtin_amdgcn_raw_buffer_load_b64(rxp, (uint32_t)(t * K + r) * 2u, 0, kCoherent);
                else
                    x2 = *(const u32x2 *)(xp + (size_t)t * K + r);
                v.x[t][0] = x2[0];
                v.x[t][1] = x2[1];
            } else {
                const int r = r0 < nrows ? r0 : 0;
                if constexpr (CX)
                    v.x[t][0] = __builtin_amdgcn_raw_buffer_load_b32(rxp, (uint32_t)(t * K + r) * 2u, 0, kCoherent);
                else
                    v.x[t][0] = *(const uint32_t *)(xp + (size_t)t * K + r);
            }
        }
    };
    auto load_w = [&](Batch &v, int b) __attribute__((always_inline)) {
        const int r0 = (RG * b + rg) * U;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = min(r0 + u, nrows - 1);
#pragma unroll
            for (int w = 0; w < NW; ++w)
                v.w[u][w] = __builtin_nontemporal_load((const u32x4 *)(wp[w] + (size_t)r * M));
        }
    };
    auto load_batch = [&](Batch &v, int b) __attribute__((always_inline)) {
        load_x(v, b);
        // The activations must be issued before the weights: loads complete
        // in order, so waiting for a batch's weights then covers them too.
        __builtin_amdgcn_sched_barrier(0);
        load_w(v, b);
    };
    constexpr int DEPTH = gemv_depth<NT>();
    const int nb = (nrows + RG * U - 1) / (RG * U);
    Batch ring[DEPTH];
    bool ready = true; // block-uniform
    // Prologue: DEPTH batches (past the split if i >= nb: never accumulated).
    if constexpr (CX) {
#pragma unroll
        for (int i = 0; i < DEPTH; ++i)
            load_w(ring[i], i);
        ready = wait();
#pragma unroll
        for (int i = 0; i < DEPTH; ++i)
            load_x(ring[i], i);
    } else {
#pragma unroll
        for (int i = 0; i < DEPTH; ++i)
            load_batch(ring[i], i);
    }

    float acc[NW][NT][8];
    float ssq[NT]; // RMS: this row group's sum of x^2 per token
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int e = 0; e < 8; ++e)
                acc[w][t][e] = 0.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t)
        ssq[t] = 0.0f;

    {
        auto fma_batch = [&](const Batch &bt, int b) __attribute__((always_inline)) {
            const int r0 = (RG * b + rg) * U;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (r0 + u < nrows) {
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        const float x = u & 1 ? bf16_hi(bt.x[t][u / 2]) : bf16_lo(bt.x[t][u / 2]);
                        if constexpr (RMS)
                            ssq[t] += x * x;
#pragma unroll
                        for (int w = 0; w < NW; ++w)
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                acc[w][t][2 * e] += x * bf16_lo(bt.w[u][w][e]);
                                acc[w][t][2 * e + 1] += x * bf16_hi(bt.w[u][w][e]);
                            }
                    }
                }
            }
        };
        // Steady state: DEPTH batches in flight, loads unconditional.  Batch
        // b lives in ring[b % DEPTH].
        int b = 0;
        for (; b + 2 * DEPTH - 1 < nb; b += DEPTH) {
#pragma unroll
            for (int i = 0; i < DEPTH; ++i) {
                fma_batch(ring[i], b + i);
                load_batch(ring[i], b + i + DEPTH);
            }
        }
        // The last 1 .. 2*DEPTH-1 batches.
#pragma unroll
        for (int i = 0; i < DEPTH; ++i) {
            if (b + i < nb)
                fma_batch(ring[i], b + i);
            if (b + i + DEPTH < nb)
                load_batch(ring[i], b + i + DEPTH);
        }
#pragma unroll
        for (int i = 0; i < DEPTH; ++i)
            if (b + i + DEPTH < nb)
                fma_batch(ring[i], b + i + DEPTH);
    }

    // Half-wave row groups: groups 2*wave and 2*wave+1 share columns, so
    // the two wave halves are added first.  (With 1 KB segments every lane
    // of a wave reads the same rows.)
    if constexpr (L::HALVES == 2) {
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    acc[w][t][e] += __shfl_xor(acc[w][t][e], 32);
        if constexpr (RMS)
#pragma unroll
            for (int t = 0; t < NT; ++t)
                ssq[t] += __shfl_xor(ssq[t], 32);
    }
    if constexpr (RMS)
        if (lane == 0)
#pragma unroll
            for (int t = 0; t < NT; ++t)
                sh.ssq[wave][t] = ssq[t];
    if (lane < L::LANES) {
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                f32x4 lo = {acc[w][t][0], acc[w][t][1], acc[w][t][2], acc[w][t][3]};
                f32x4 hi = {acc[w][t][4], acc[w][t][5], acc[w][t][6], acc[w][t][7]};
                *(f32x4 *)&sh.red[wave][w][t][col] = lo;
                *(f32x4 *)&sh.red[wave][w][t][col + 4] = hi;
            }
    }
    __syncthreads();

    // Thread tid < STRIP now owns column m0 + tid of the strip (threads past
    // the strip, in blocks with more threads than columns, sum column 0 and
    // store nothing); the waves' sums are added in wave order.
    const int m = m0 + tid;
    const bool mvalid = tid < width && m < M;
    const int c = tid < L::STRIP ? tid : 0;
    float v[NW][NT];
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            float s = sh.red[0][w][t][c];
#pragma unroll
            for (int q = 1; q < L::WAVES; ++q)
                s += sh.red[q][w][t][c];
            v[w][t] = s;
        }
    if (!ready)
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int t = 0; t < NT; ++t)
                v[w][t] = __builtin_nanf("");
    float ss[NT]; // RMS: the block's (then the whole row's) sum of x^2 per token
    if constexpr (RMS)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            float s = sh.ssq[0][t];
#pragma unroll
            for (int q = 1; q < L::WAVES; ++q)
                s += sh.ssq[q][t];
            ss[t] = s;
        }

    if (p.splits > 1) {
        // Per-item sums go out with device-coherent stores; once they have
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
        // Every strip of a split sums the same rows' x^2: each strip keeps
        // its own copy, so no two blocks store to the same word.
        if constexpr (RMS)
            if (tid < NT)
                __hip_atomic_store(&p.ssq[(strip * p.splits + split) * NT + tid], ss[tid], __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        wait_vmcnt<0>();
        __syncthreads();
        if (tid == 0) {
            const uint32_t before =
                __hip_atomic_fetch_add(p.counters + p.counter_stride * strip, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            sh.last = before == (uint32_t)(p.splits - 1);
        }
        __syncthreads();
        if (!sh.last)
            return false;
        if (tid == 0)
            __hip_atomic_store(p.counters + p.counter_stride * strip, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (mvalid) {
            // Sum the splits in order 0, 1, 2, ...; the loads of C splits are
            // in flight at once (with RMSNorm, their sums of x^2 too, added
            // the same way).  They are unconditional (a slot past the last
            // split reloads this block's own), so there are no branches; the
            // values past the last split are not added.
            constexpr int C = gemv_reduce_batch<NT, NW>();
            const size_t stride = (size_t)NW * NT * M;
            const float *src = &p.partial[m];
            float sum[NW][NT], tot[NT];
            for (int s0 = 0; s0 < p.splits; s0 += C) {
                float x[C][NW][NT], q[C][NT];
#pragma unroll
                for (int u = 0; u < C; ++u) {
                    const int sp = s0 + u < p.splits ? s0 + u : split;
#pragma unroll
                    for (int w = 0; w < NW; ++w)
#pragma unroll
                        for (int t = 0; t < NT; ++t)
                            x[u][w][t] = __hip_atomic_load(src + sp * stride + ((size_t)w * NT + t) * M,
                                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if constexpr (RMS)
#pragma unroll
                        for (int t = 0; t < NT; ++t)
                            q[u][t] = __hip_atomic_load(&p.ssq[(strip * p.splits + sp) * NT + t],
                                                        __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
#pragma unroll
                for (int u = 0; u < C; ++u) {
                    const int sp = s0 + u;
#pragma unroll
                    for (int w = 0; w < NW; ++w)
#pragma unroll
                        for (int t = 0; t < NT; ++t) {
                            const float xv = sp == split ? v[w][t] : x[u][w][t];
                            sum[w][t] = sp == 0 ? xv : sp < p.splits ? sum[w][t] + xv : sum[w][t];
                        }
                    if constexpr (RMS)
#pragma unroll
                        for (int t = 0; t < NT; ++t) {
                            const float qv = sp == split ? ss[t] : q[u][t];
                            tot[t] = sp == 0 ? qv : sp < p.splits ? tot[t] + qv : tot[t];
                        }
                }
            }
#pragma unroll
            for (int w = 0; w < NW; ++w)
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    v[w][t] = sum[w][t];
            if constexpr (RMS)
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    ss[t] = tot[t];
        }
    }

    if (mvalid) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            float y;
            if constexpr (EPI == EPI_GATE_MUL) {
                float g = v[0][t], u = v[NW - 1][t];
                if constexpr (RMS) {
                    const float r = 1.0f / __builtin_sqrtf(ss[t] / (float)K + p.eps);
                    g *= r;
                    u *= r;
                }
                y = gate_act(g, p.activation, p.beta) * u;
            } else {
                y = v[0][t];
                if (p.rowdiv)
                    y = y / p.rowdiv[t];
            }
            const uint16_t bits = __builtin_bit_cast(uint16_t, (__bf16)y);
            if constexpr (CO)
                __builtin_amdgcn_raw_buffer_store_b16(bits, make_rsrc(p.out), (uint32_t)(t * M + m) * 2u, 0,
                                                      kCoherent);
            else
                p.out[(size_t)t * M + m] = bits;
        }
    }
    return true;
}

// At most 256 VGPRs per lane: two 4-wave blocks per CU stay resident.
template <int NT, int NW, int EPI, bool RMS = false>
__global__ __launch_bounds__((GemvLayout<NT, NW>::THREADS)) __attribute__((amdgpu_waves_per_eu(2)))
void gemv_splitk_kernel(GemvParams p)
{
    __shared__ GemvShared<NT, NW> sh;
    gemv_item<NT, NW, EPI, RMS>(p, blockIdx.x, sh);
}

// ---- one kernel for both steps (decode, T <= 8) -------------------------------

struct GemvFusedParams {
    GemvParams gate_up, down;    // down.counters must not overlap gate_up.counters
    uint32_t *ready;             // per down split s, word [kFlagStride*s] (zero on entry and exit):
                                 // gate/up strips done that it reads, plus kConsumerUnit per down
                                 // block of the split past its wait
    uint32_t *errors;            // count of down blocks whose wait gave up (sticky: the host clears it)
    uint32_t spin_limit;         // polls before a waiting block gives up
};

// What a down block adds to its split's ready word once past its wait; the
// gate/up strips a split reads (at most kMaxDim / 256 = 16384) stay in the
// low 16 bits, and down blocks per split (as many) times this unit below 2^31.
constexpr uint32_t kConsumerUnit = 1u << 16;

// Gate/up strips (of 8 * strip_lanes columns of H) that overlap the rows
// [s * k_split, (s + 1) * k_split) of down split s.
__device__ __forceinline__ uint32_t fused_strips_of_split(const GemvParams &gu, const GemvParams &dn, int s)
{
    const int width = 8 * gu.strip_lanes;
    const int r0 = s * dn.k_split, r1 = min(dn.K, r0 + dn.k_split);
    return (uint32_t)((r1 - 1) / width - r0 / width + 1);
}

// Add `delta` to a split's ready word; the add that completes the split's
// events of this call (every gate/up strip it reads and every down block
// past its wait: need + consumers * kConsumerUnit in all) resets the word
// to zero.  Exactly one add completes it, and none follows, so the word is
// zero when the kernel ends whatever order the adds land in.
__device__ __forceinline__ void fused_ready_add(uint32_t *w, uint32_t delta, uint32_t complete)
{
    const uint32_t old = __hip_atomic_fetch_add(w, delta, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old + delta == complete)
        __hip_atomic_store(w, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// What a down block waits for: every gate/up strip its split reads is
// written (the low half of the split's ready word reaches `need`).  Thread 0
// polls the split's own line.  Only blocks of lower index (dispatched
// earlier) are waited for, so the wait ends whatever number of blocks the
// device holds at once; a block that polls spin_limit times gives up: it
// counts itself in `errors` and its sums become NaN (gemv_item), so the
// strips of Y it feeds are NaN, never silently wrong.  Either way it adds
// its kConsumerUnit, so the word still returns to zero.
struct FusedWait {
    uint32_t *w;         // the split's ready word
    uint32_t need;       // gate/up strips the split reads
    uint32_t consumers;  // down blocks of the split (its strips of Y)
    uint32_t spin_limit;
    uint32_t *errors;
    __device__ bool operator()() const
    {
        __shared__ int s_ready;
        if (threadIdx.x == 0) {
            uint32_t v = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            for (uint32_t polls = 0; (v & (kConsumerUnit - 1)) < need && polls < spin_limit; ++polls) {
                __builtin_amdgcn_s_sleep(2);
                v = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            const bool ready = (v & (kConsumerUnit - 1)) >= need;
            fused_ready_add(w, kConsumerUnit, need + consumers * kConsumerUnit);
            if (!ready)
                __hip_atomic_fetch_add(errors, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_ready = ready;
        }
        wait_lgkm0(); // thread 0's LDS write lands before the barrier
        barrier_only();
        return s_ready != 0;
    }
};

// The whole Gated MLP for T <= 8 in one launch of n_gu + n_dn blocks:
// blocks below n_gu run the gate/up items (H written through to memory with
// device-coherent stores); the block that completes a strip of H then
// counts it in for every down split that reads it.  The other blocks run the
// down items: they issue their first weight loads, wait for their split's
// strips of H, and read H with device-coherent loads.  Items and reductions
// are those of the two-kernel GEMV path, so Y is bit for bit that path's.
template <int NT, bool RMS>
__global__ __launch_bounds__((GemvLayout<NT, 2>::THREADS)) __attribute__((amdgpu_waves_per_eu(2)))
void gemv_fused_kernel(GemvFusedParams p)
{
    static_assert(GemvLayout<NT, 2>::THREADS == GemvLayout<NT, 1>::THREADS, "one block size for both steps");
    __shared__ union {
        GemvShared<NT, 2> gate_up;
        GemvShared<NT, 1> down;
    } sh;
    const int n_gu = p.gate_up.strips * p.gate_up.splits;
    const uint32_t consumers = (uint32_t)p.down.strips;
    const int b = blockIdx.x;
    if (b < n_gu) {
        if (gemv_item<NT, 2, EPI_GATE_MUL, RMS, true>(p.gate_up, b, sh.gate_up)) {
            wait_vmcnt<0>(); // this wave's part of the strip is written through
            __syncthreads();
            if (threadIdx.x == 0) {
                const int width = 8 * p.gate_up.strip_lanes;
                const int j = b % p.gate_up.strips;
                const int f0 = j * width, f1 = min(p.gate_up.M, f0 + width);
                for (int s = f0 / p.down.k_split; s <= (f1 - 1) / p.down.k_split; ++s)
                    fused_ready_add(p.ready + kFlagStride * s, 1u,
                                    fused_strips_of_split(p.gate_up, p.down, s) + consumers * kConsumerUnit);
            }
        }
        return;
    }
    const int item = b - n_gu;
    const int split = item / p.down.strips;
    const FusedWait wait{p.ready + kFlagStride * split, fused_strips_of_split(p.gate_up, p.down, split),
                         consumers, p.spin_limit, p.errors};
    gemv_item<NT, 1, EPI_STORE, false, false, true>(p.down, item, sh.down, wait);
}

} // namespace gmlp
