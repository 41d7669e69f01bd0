// The whole Gated MLP in one launch of the MFMA GEMM kernels, for few tokens
// (one token tile: T <= 64).
//
// The paper's deepest fusion keeps the intermediate of a multi-operator
// kernel on chip (loop fusion, Section 4.5; the fusion ablation of Section
// 6.4).  On this GPU a block's LDS (160 KB) cannot hold a token tile's whole
// row of H, so H still passes through memory; what one launch removes is the
// boundary between the two GEMMs (the drain of the first and the ramp of the
// second).  Blocks below n_gu run the gate/up tiles of the two-kernel plan;
// the block that writes a tile of H (the last of its splits) writes it with
// device-coherent stores and then counts it in for every down split whose
// rows of H it covers.  The other blocks run the down tiles: before loading
// any H they wait until their split's count is complete (FusedWait, the same
// bounded wait and ready-word protocol as the decode kernel), then read H
// with device-coherent loads.  A down block waits only for gate/up blocks,
// whose indices are lower (the hardware dispatches them first) and which
// never wait, so no co-residency is needed.  Tiles, splits and reduction
// orders are the two-kernel plan's, so Y is that plan's bit for bit.
#pragma once

#include "gemm_mfma.hpp"
#include "gemv.hpp"

namespace gmlp {

struct GemmFusedParams {
    GemmParams gate_up, down; // one token tile each; down's counters and partial sums after gate/up's
    uint32_t *ready;          // per down split s, word [kFlagStride * s] (zero on entry and exit)
    uint32_t *errors;         // count of down blocks whose wait gave up (sticky: the host clears it)
    uint32_t spin_limit;      // polls before a waiting block gives up
};

// Gate/up tiles (of GU::BMW columns of H) overlapping the rows
// [s * k_split, (s + 1) * k_split) of down split s.
template <class GU>
__device__ __forceinline__ uint32_t fused_gemm_tiles_of_split(const GemmParams &dn, int s)
{
    const int r0 = s * dn.k_split, r1 = min(dn.K, r0 + dn.k_split);
    return (uint32_t)((r1 - 1) / GU::BMW - r0 / GU::BMW + 1);
}

// Bytes of LDS stage i of the fused kernel: the larger of the two steps'
// stage i (16 where neither step has one).
template <class GU, class DN>
constexpr int fused_stage_bytes(int i)
{
    const int g = i < GU::STAGES ? GU::STAGE_BYTES : 16, d = i < DN::STAGES ? DN::STAGE_BYTES : 16;
    return g > d ? g : d;
}

template <class GU, class DN>
constexpr int fused_lds_bytes()
{
    int n = 0;
    for (int i = 0; i < 8; ++i)
        n += fused_stage_bytes<GU, DN>(i);
    return n;
}

template <class GU, class DN>
__global__ __launch_bounds__(GU::NTHREADS, 1) void gemm_fused_kernel(GemmFusedParams fp)
{
    static_assert(GU::NTHREADS == DN::NTHREADS, "one block size for both steps");
    static_assert(GU::STAGES <= 8 && DN::STAGES <= 8, "at most 8 stages");
    static_assert(fused_lds_bytes<GU, DN>() + 512 <= 160 * 1024, "LDS capacity of a CU");
    // One LDS array per stage, as in gemm_mfma_kernel (distinct objects let
    // the compiler see that the DMA into one stage does not alias the reads
    // of another; a single shared buffer makes it drain the ring at every
    // k-tile).  A block runs one of the two steps, so stage i of both steps
    // shares array i.
    __shared__ __attribute__((aligned(1024))) uint8_t lds0[fused_stage_bytes<GU, DN>(0)];
    __shared__ __attribute__((aligned(1024))) uint8_t lds1[fused_stage_bytes<GU, DN>(1)];
    __shared__ __attribute__((aligned(1024))) uint8_t lds2[fused_stage_bytes<GU, DN>(2)];
    __shared__ __attribute__((aligned(1024))) uint8_t lds3[fused_stage_bytes<GU, DN>(3)];
    __shared__ __attribute__((aligned(1024))) uint8_t lds4[fused_stage_bytes<GU, DN>(4)];
    __shared__ __attribute__((aligned(1024))) uint8_t lds5[fused_stage_bytes<GU, DN>(5)];
    __shared__ __attribute__((aligned(1024))) uint8_t lds6[fused_stage_bytes<GU, DN>(6)];
    __shared__ __attribute__((aligned(1024))) uint8_t lds7[fused_stage_bytes<GU, DN>(7)];
    auto stage = [&](auto s) __attribute__((always_inline)) -> uint8_t * {
        if constexpr (decltype(s)::value == 0) return lds0;
        else if constexpr (decltype(s)::value == 1) return lds1;
        else if constexpr (decltype(s)::value == 2) return lds2;
        else if constexpr (decltype(s)::value == 3) return lds3;
        else if constexpr (decltype(s)::value == 4) return lds4;
        else if constexpr (decltype(s)::value == 5) return lds5;
        else if constexpr (decltype(s)::value == 6) return lds6;
        else return lds7;
    };
    const int n_gu = fp.gate_up.tile_count * fp.gate_up.splits;
    const uint32_t consumers = (uint32_t)fp.down.tile_count;
    const int b = blockIdx.x;
    if (b < n_gu) {
        const int m0 = gemm_block<GU, EPI_GATE_MUL, true, true, 0, kCoherent>(fp.gate_up, b, stage);
        if (m0 >= 0) { // this block wrote H[:, m0 : m0 + BMW]
            wait_vmcnt<0>(); // this wave's stores of the tile are written through
            __syncthreads();
            if (threadIdx.x == 0) {
                const int ks = fp.down.k_split;
                const int f1 = min(fp.gate_up.M, m0 + GU::BMW);
                for (int s = m0 / ks; s <= (f1 - 1) / ks; ++s)
                    fused_ready_add(fp.ready + kFlagStride * s, 1u,
                                    fused_gemm_tiles_of_split<GU>(fp.down, s) + consumers * kConsumerUnit);
            }
        }
        return;
    }
    const int j = b - n_gu;
    const int split = gemm_split_of_block(fp.down, j);
    const FusedWait wait{fp.ready + kFlagStride * split, fused_gemm_tiles_of_split<GU>(fp.down, split), consumers,
                         fp.spin_limit, fp.errors};
    gemm_block<DN, EPI_STORE, true, true, kCoherent, 0>(fp.down, j, stage, wait);
}

} // namespace gmlp
