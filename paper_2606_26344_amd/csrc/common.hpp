// Shared device-side types and helpers of the gfx950 Gated MLP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gmlp {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short i16x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

// What the last step of a kernel writes.
enum Epilogue {
    EPI_GATE_MUL = 0, // out = bf16(act(acc0) * acc1)    (H of the gate/up step)
    EPI_STORE = 1,    // out = bf16(acc0)                (Y of the down step)
    EPI_GATE_PAIR = 2, // out = bf16(act(G) * U), G and U from the two blocks of a pair
};

#define GMLP_LDS(p) ((__attribute__((address_space(3))) void *)(p))

// Buffer-resource word 3 for raw (untyped, stride 0) buffers on gfx9 parts.
constexpr int kRawBufferWord3 = 0x00020000;
// A byte offset no buffer in this library reaches: loads at it are out of
// range and return zeros (used to zero-fill tile edges).
constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int kNumRecords = 0x7fffffff;
// Cache-policy operand of the buffer load/store builtins for device-coherent
// (agent-scope) accesses on gfx950: the SC1 bit, the same policy the compiler
// gives agent-scope atomic loads and stores.
constexpr int kCoherent = 16;
// Cache-policy operand for streaming (nontemporal) loads: the NT bit.
constexpr int kNonTemporal = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, kNumRecords,
                                             kRawBufferWord3);
}

// 16 bytes from global memory (resource + voff + soff bytes) straight into
// LDS.  Lane i of the wave writes lds_wave_base + 16 * i; lds_wave_base and
// soff must be the same for every lane of the wave.  A lane whose voff is
// kOutOfRange reads zeros (soff stays far below 2^31, so voff + soff cannot
// wrap back into range).
__device__ __forceinline__ void load16_to_lds(__amdgpu_buffer_rsrc_t r, void *lds_wave_base,
                                              uint32_t voff, uint32_t soff = 0)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, GMLP_LDS(lds_wave_base), 16, voff, soff, 0, 0);
}

// As load16_to_lds, with the nontemporal (streaming) cache policy: for data
// that is read exactly once, so that it does not displace reused lines.
__device__ __forceinline__ void load16_to_lds_stream(__amdgpu_buffer_rsrc_t r, void *lds_wave_base,
                                                     uint32_t voff, uint32_t soff = 0)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, GMLP_LDS(lds_wave_base), 16, voff, soff, 0, kNonTemporal);
}

// Wait until at most n vector-memory operations of this wave are in flight
// (gfx9 s_waitcnt encoding: vmcnt split over bits [3:0] and [15:14]; expcnt
// and lgkmcnt left at their "no wait" maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit field");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Wait for this wave's outstanding LDS reads (lgkmcnt = 0) only.
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// Workgroup barrier that, unlike __syncthreads(), does not also wait for
// every outstanding global load of the wave (which would drain the LDS DMA
// prefetch ring).  Callers wait for exactly what they need first.  The empty
// asm statements keep the compiler from moving memory accesses across it.
__device__ __forceinline__ void barrier_only()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// fp32 -> bf16 with round-to-nearest-even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    uint16_t a = __builtin_bit_cast(uint16_t, (__bf16)lo);
    uint16_t b = __builtin_bit_cast(uint16_t, (__bf16)hi);
    return (uint32_t)a | ((uint32_t)b << 16);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xffff0000u); }

// silu(z) = z * sigmoid(z) = z / (1 + e^-z) in fp32.  For z << 0, e^-z
// overflows to +inf and the reciprocal to 0, giving -0 (the exact value is
// below fp32's smallest normal there).
__device__ __forceinline__ float silu(float z)
{
    return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

// Gate activations of the Gated MLP family (values of enum gmlp_activation).
enum Activation {
    ACT_SILU = 0,    // silu(g)                    the SiLU Gated MLP
    ACT_SWISH = 1,   // g * sigmoid(beta * g)      the SwiGLU Gated MLP
    ACT_SIGMOID = 2, // sigmoid(g)                 the GLU Gated MLP
};

// act(g) for a block-uniform activation, without branches:
// act(g) = a * sigmoid(beta * g) with a = g for silu and swish_beta and a = 1
// for sigmoid.  The caller passes beta = 1 for silu and sigmoid, where the
// product beta * g is then exactly g, so this is silu(g) bit for bit.
__device__ __forceinline__ float gate_act(float g, int act, float beta)
{
    const float s = __builtin_amdgcn_rcpf(1.0f + __expf(-(beta * g)));
    return (act == ACT_SIGMOID ? 1.0f : g) * s;
}

// Hardware places consecutive workgroups round-robin on the 8 XCDs (each with
// its own L2).  Renumber them so each XCD receives one contiguous range of
// the logical tile order; neighbouring tiles, which share operand strips,
// then share an L2.  A bijection on [0, n) whatever the placement.
__device__ __forceinline__ int xcd_contiguous_id(int bid, int n)
{
    const int xcd = bid & 7, j = bid >> 3;
    const int q = n >> 3, r = n & 7;
    return (xcd < r ? xcd * (q + 1) : r * (q + 1) + (xcd - r) * q) + j;
}

} // namespace gmlp
