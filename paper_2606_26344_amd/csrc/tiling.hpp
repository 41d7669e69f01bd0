// Tile shapes and work-item constants of the Gated MLP kernels, shared by the
// kernels (gemm_mfma.hpp, gemv.hpp) and the host-side planning (plan.hpp).
// Plain C++: no HIP dependency.
#pragma once

namespace gmlp {

// A configuration of gemm_mfma_kernel: NW weights sharing each activation
// tile (2 for gate/up, 1 for down), a WM x WN grid of waves, each wave
// holding TM x TN MFMA tiles of 32 x 32 outputs per weight, a ring of STAGES
// LDS stages of BK rows of k.
template <int NW_, int WM_, int WN_, int TM_, int TN_, int STAGES_, int BK_>
struct GemmShape {
    static constexpr int NW = NW_, WM = WM_, WN = WN_, TM = TM_, TN = TN_, STAGES = STAGES_;
    static constexpr int BK = BK_;
    // The MFMA instruction: tiles of 256 tokens or 256 columns (the
    // MFMA-bound prefill tiles) issue v_mfma_f32_16x16x32_bf16, four 16 x 16
    // accumulators per 32 x 32 block in k32 steps; under the board's power
    // cap it sustains 15% more than v_mfma_f32_32x32x16_bf16 on random
    // operands, and the steps on those tiles ran 0.6-2.6% faster with it
    // (T = 640..4096 at D = 4096, F = 14336, and the large-prefill shape, on
    // two boards).  The smaller tiles, bound by the weight stream, keep
    // 32x32x16 in k16 steps (16x16x32 was 1-4% slower there).
    static constexpr bool M16 = BK == 64 && (WM * TM * 32 >= 256 || WN * TN * 32 >= 256);
    static constexpr int MFMA_K = M16 ? 32 : 16;
    static constexpr int KSTEPS = BK / MFMA_K;     // MFMA k steps per k-tile
    static constexpr int NWAVES = WM * WN;
    static constexpr int NTHREADS = NWAVES * 64;
    static constexpr int BMW = WM * TM * 32;       // columns per weight per tile
    static constexpr int BN = WN * TN * 32;        // tokens per tile
    static constexpr int W_ROW_BYTES = BMW * 2;    // one k row of a weight tile
    static constexpr int W_CPR = BMW / 8;          // 16-byte chunks per weight row
    static constexpr int W_TILE_BYTES = BK * BMW * 2;
    // Activation tiles are stored as 128-byte LDS rows of 8 chunks.  With
    // BK = 32 one token row is 4 chunks, so row r holds token r in chunks
    // 0..3 and token r + BN/2 in chunks 4..7.
    static constexpr int X_HALVES = 128 / (BK * 2); // tokens per 128-byte LDS row
    static constexpr int X_ROWS = BN / X_HALVES;    // LDS rows of an activation tile
    static constexpr int X_CPT = BK / 8;            // 16-byte chunks per token
    static constexpr int X_TILE_BYTES = BN * BK * 2;
    static constexpr int STAGE_BYTES = NW * W_TILE_BYTES + X_TILE_BYTES;
    static constexpr int W_LOADS = W_TILE_BYTES / (NTHREADS * 16); // per weight, per thread
    static constexpr int X_LOADS = X_TILE_BYTES / (NTHREADS * 16);
    static constexpr int LOADS_PER_STAGE = NW * W_LOADS + X_LOADS;
    static constexpr int W_LPR = 64 / W_CPR;          // weight rows per wave load
    static constexpr int W_RPI = NWAVES * W_LPR;      // weight rows per load step i
    // LDS reads and MFMAs per k step (a 32 x 32 block per MFMA, or 16 x 16
    // subtiles: twice the reads per step of twice the k, four MFMAs).
    static constexpr int FRAG_READS = M16 ? NW * TM * 4 + TN * 2 : NW * TM * 2 + TN;
    static constexpr int MFMAS = M16 ? NW * TM * TN * 4 : NW * TM * TN;
    static_assert(BK == 32 || BK == 64, "k-tile of 32 or 64");
    static_assert(X_ROWS % 32 == 0, "n-tiles of 32 tokens do not straddle the two row halves");
    static_assert(BMW >= 64, "weight rows of at least 8 chunks");
    static_assert(W_TILE_BYTES % (NTHREADS * 16) == 0 && X_TILE_BYTES % (NTHREADS * 16) == 0,
                  "every thread issues whole 16-byte loads");
    static_assert(STAGES >= 2 && STAGES <= 8, "2..8 LDS stages");
    static_assert((STAGES - 2) * LOADS_PER_STAGE < 64, "vmcnt range");
    static_assert(STAGES * STAGE_BYTES + 256 <= 160 * 1024, "LDS capacity of a CU (with the kernel's other shared words)");
};

// ---- split-K GEMV (T <= 8) ---------------------------------------------------
// Block layouts.  Up to kGemvWideTokens tokens a block is 8 waves; the
// gate/up step (two weights) gives each wave one 1 KB segment of a weight
// row per load (64 lanes x 8 columns: 512-column strips, 8 row groups) and
// the down step each 32-lane half of a wave a 512-byte segment (256-column
// strips, 16 row groups).  Above, a block is 4 waves of 512-byte half-wave
// segments (256-column strips, 8 row groups), which leaves the registers for
// the accumulators of more tokens and lets two blocks share a CU.  Measured
// on MI355X at D = 4096, F = 14336, same process: T = 1 step 59.3 against
// 60.0 us (gate/up 37.4 against 38.2), T = 2 61.3 against 62.0, but T = 4
// 64.1 against 62.8; for the down step 1 KB segments were slower (T = 1:
// 21.8 against 21.3 us).
constexpr int kGemvWideTokens = 2;
template <int NT, int NW>
struct GemvLayout {
    static constexpr int THREADS = NT <= kGemvWideTokens ? 512 : 256;
    static constexpr int LANES = NT <= kGemvWideTokens && NW == 2 ? 64 : 32; // lanes per row segment
    static constexpr int STRIP = 8 * LANES;        // columns per strip, one per thread at most
    static constexpr int WAVES = THREADS / 64;
    static constexpr int RG = THREADS / LANES;     // row groups
    static constexpr int HALVES = 64 / LANES;      // row groups per wave
    static_assert(STRIP <= THREADS, "one column per thread in the reduction");
};
// Threads and lanes per row segment of the GEMV blocks (host side).
constexpr int gemv_threads(int nt) { return nt <= kGemvWideTokens ? 512 : 256; }
constexpr int gemv_strip_lanes(int nt, int nw) { return nt <= kGemvWideTokens && nw == 2 ? 64 : 32; }

// Weight rows per lane per load batch (U), and batches in flight per lane
// (DEPTH): DEPTH*NW*U loads of 16 bytes in flight per lane, within the
// register budget of NT tokens (with the 512-thread blocks, 128 KB in flight
// per block at U = 4 for the gate/up step).  The down step's 8-wave blocks
// (up to kGemvWideTokens tokens) do best with less in flight: U = 2, i.e.
// 32 KB per block (measured at D = 4096, F = 14336: down 20.4 -> 19.9 us at
// T = 1, 20.9 -> 20.6 at T = 2; U = 2 for the 4-wave blocks of T = 3..5 was
// 25-29% slower, and a third batch in flight at U = 4 made T = 1 23.6 us).
template <int NT, int NW>
constexpr int gemv_batch_rows() { return NW == 1 && NT <= kGemvWideTokens ? 2 : NT <= 6 ? 4 : 2; }
template <int NT>
constexpr int gemv_depth() { return 2; }

// The fused decode kernel: at most this many down splits, each with a ready
// word on its own 128-byte line.
constexpr int kFusedMaxSplits = 512;
constexpr int kFlagStride = 32; // words between the ready words of two splits: one 128-byte line each

} // namespace gmlp
