// mfma_ceiling: the sustained bf16 matrix-core rate of this board, for the
// roofline context of the MFMA-bound Gated MLP steps.
//
// Every SIMD runs two waves that issue MFMAs back to back on register
// operands (no memory traffic in the loop): v_mfma_f32_32x32x16_bf16 (the
// GEMM kernels' instruction, 8 independent accumulators per wave) and
// v_mfma_f32_16x16x32_bf16 (16 accumulators, the same FLOPs per loop), each
// once with operands drawn from a uniform random distribution and once with
// all-zero operands.  The board's power limit makes the random-data rate the
// ceiling any GEMM on random data can reach with that instruction; the
// zero-data rate shows the clock-limited peak.  Prints one JSON object per
// run on stdout.
//
//     mfma_ceiling [milliseconds per run, default 20]
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kBlocks = 256;  // one per CU
constexpr int kThreads = 512; // two waves per SIMD
constexpr int kAcc = 8;       // independent accumulators per wave
constexpr int kOperands = 1 << 16;
constexpr double kFlopPerMfma = 2.0 * 32 * 32 * 16;
constexpr double kNominalTflops = 2516.6; // 256 CUs x 4096 FLOP/clk x 2.4 GHz

// One loop iteration is kAcc x 32768 FLOP per wave with either instruction.
template <bool M16>
__global__ __launch_bounds__(kThreads, 1) void mfma_loop(const bf16x8 *src, float *out, int iters)
{
    const int tid = blockIdx.x * blockDim.x + threadIdx.x;
    const bf16x8 a0 = src[(4 * tid) % kOperands], a1 = src[(4 * tid + 1) % kOperands];
    const bf16x8 b0 = src[(4 * tid + 2) % kOperands], b1 = src[(4 * tid + 3) % kOperands];
    float s = 0.0f;
    if constexpr (M16) {
        f32x4 acc[2 * kAcc];
        for (int i = 0; i < 2 * kAcc; ++i)
            acc[i] = f32x4{};
        for (int it = 0; it < iters; ++it) {
#pragma unroll
            for (int i = 0; i < 2 * kAcc; ++i)
                acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16((i & 1) ? a1 : a0, (i & 2) ? b1 : b0, acc[i], 0, 0,
                                                                 0);
        }
        for (int i = 0; i < 2 * kAcc; ++i)
            for (int e = 0; e < 4; ++e)
                s += acc[i][e];
    } else {
        f32x16 acc[kAcc];
        for (int i = 0; i < kAcc; ++i)
            acc[i] = f32x16{};
        for (int it = 0; it < iters; ++it) {
#pragma unroll
            for (int i = 0; i < kAcc; ++i)
                acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16((i & 1) ? a1 : a0, (i & 2) ? b1 : b0, acc[i], 0, 0,
                                                                 0);
        }
        for (int i = 0; i < kAcc; ++i)
            for (int e = 0; e < 16; ++e)
                s += acc[i][e];
    }
    out[tid] = s; // keeps the loop live
}

int check(hipError_t e, const char *what)
{
    if (e != hipSuccess) {
        fprintf(stderr, "mfma_ceiling: %s: %s\n", what, hipGetErrorString(e));
        exit(1);
    }
    return 0;
}

} // namespace

int main(int argc, char **argv)
{
    const double target_ms = argc > 1 ? atof(argv[1]) : 20.0;
    if (!(target_ms > 0.0 && target_ms <= 1000.0)) {
        fprintf(stderr, "usage: mfma_ceiling [milliseconds per run, 0 < ms <= 1000]\n");
        return 2;
    }
    // Uniform values in [-1, 1), rounded to bf16 by truncation (any spread
    // of mantissa bits does: what matters is that the operands toggle).
    std::vector<uint16_t> host(kOperands * 8);
    uint32_t x = 12345u;
    for (auto &v : host) {
        x = x * 1664525u + 1013904223u;
        const float f = ((int)(x >> 9) - (1 << 22)) / (float)(1 << 22);
        uint32_t bits;
        std::memcpy(&bits, &f, sizeof bits);
        v = (uint16_t)(bits >> 16);
    }
    bf16x8 *rnd = nullptr, *zero = nullptr;
    float *out = nullptr;
    check(hipMalloc(&rnd, sizeof(bf16x8) * kOperands), "hipMalloc");
    check(hipMalloc(&zero, sizeof(bf16x8) * kOperands), "hipMalloc");
    check(hipMalloc(&out, sizeof(float) * kBlocks * kThreads), "hipMalloc");
    check(hipMemcpy(rnd, host.data(), sizeof(bf16x8) * kOperands, hipMemcpyHostToDevice), "hipMemcpy");
    check(hipMemset(zero, 0, sizeof(bf16x8) * kOperands), "hipMemset");
    hipEvent_t e0, e1;
    check(hipEventCreate(&e0), "hipEventCreate");
    check(hipEventCreate(&e1), "hipEventCreate");
    auto run = [&](bool m16, const bf16x8 *src, int iters) {
        check(hipEventRecord(e0), "hipEventRecord");
        if (m16)
            hipLaunchKernelGGL(mfma_loop<true>, dim3(kBlocks), dim3(kThreads), 0, 0, src, out, iters);
        else
            hipLaunchKernelGGL(mfma_loop<false>, dim3(kBlocks), dim3(kThreads), 0, 0, src, out, iters);
        check(hipGetLastError(), "launch");
        check(hipEventRecord(e1), "hipEventRecord");
        check(hipEventSynchronize(e1), "hipEventSynchronize");
        float ms = 0.0f;
        check(hipEventElapsedTime(&ms, e0, e1), "hipEventElapsedTime");
        return (double)ms;
    };
    // Size the runs from a short one at the nominal clock's pace, then warm
    // up for as long as a run lasts (the power limit acts within milliseconds).
    const double probe_ms = run(false, rnd, 1000);
    const int iters = (int)std::min(2.0e6, std::max(1000.0, 1000.0 * target_ms / std::max(probe_ms, 1e-3)));
    for (int m16 = 0; m16 < 2; ++m16)
        for (int data = 0; data < 2; ++data) {
            const bf16x8 *src = data == 0 ? rnd : zero;
            run(m16, src, iters);
            const double ms = run(m16, src, iters);
            const double tflops = (double)kBlocks * (kThreads / 64) * iters * kAcc * kFlopPerMfma / ms * 1e-9;
            printf("{\"mfma\": \"%s\", \"data\": \"%s\", \"ms\": %.3f, \"tflops\": %.1f, \"frac_nominal\": %.4f, "
                   "\"iters\": %d}\n",
                   m16 ? "16x16x32" : "32x32x16", data == 0 ? "random" : "zero", ms, tflops, tflops / kNominalTflops,
                   iters);
            fflush(stdout);
        }
    check(hipFree(rnd), "hipFree");
    check(hipFree(zero), "hipFree");
    check(hipFree(out), "hipFree");
    return 0;
}
