// Host-side planning of libgmlp.so: argument validation, the tile
// configuration and launch grid of every step for a shape (the library's
// static analogue of the paper's empirical per-shape selection, Section
// 4.6), and the workspace layout.  Plain C++ with no HIP dependency, so that
// it can also be built and exercised on the host alone (the sanitizer test
// builds it with AddressSanitizer and UndefinedBehaviorSanitizer).  Included
// by one translation unit per program.
#pragma once

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <type_traits>

#include "gmlp.h"
#include "softmax_matmul.h"
#include "tiling.hpp"

namespace gmlp {
namespace {

thread_local char g_err[512];

int fail(int code, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int ok()
{
    g_err[0] = '\0';
    return GMLP_OK;
}

// ---- tile configurations -------------------------------------------------
// The large tiles run 8 waves (two per SIMD, each with half the
// accumulators), so one wave's MFMAs cover the other's waits for LDS reads,
// DMA and barriers: measured 4-7% faster than 4 waves holding the whole tile
// at T = 4096 and T = 2048 (random bf16 data; power, and so the clock, depends
// on the data at the board's power cap).
//                          NW WM WN TM TN STAGES BK
using GateUpLarge = GemmShape<2, 4, 2, 1, 4, 2, 64>; // 128 F cols x 256 tokens, per weight, 8 waves
using GateUpSmall = GemmShape<2, 4, 2, 1, 2, 3, 64>; // 128 F cols x 128 tokens, 8 waves
using DownLarge = GemmShape<1, 4, 2, 2, 4, 2, 64>;   // 256 D cols x 256 tokens, 8 waves
using DownSmall = GemmShape<1, 2, 2, 2, 2, 4, 64>;   // 128 D cols x 128 tokens
// Above 256 tokens where few down tiles fill the chip only with short
// splits: 256 x 128 tiles split over K (half the fp32 partial tile of
// DownLarge for the last block of each tile to read back).
using DownWide = GemmShape<1, 4, 2, 2, 2, 3, 64>;    // 256 D cols x 128 tokens, 8 waves
// Up to 32 tokens: the same weight tiles with one 32-token tile, so the
// activations staged per weight byte drop fourfold.
using GateUpTiny = GemmShape<2, 4, 1, 1, 1, 4, 64>; // 128 F cols x 32 tokens, 4 waves
using DownTiny = GemmShape<1, 4, 1, 1, 1, 6, 64>;   // 128 D cols x 32 tokens, 4 waves
using GateUpMid = GemmShape<2, 4, 1, 1, 2, 3, 64>;  // 128 F cols x 64 tokens, 4 waves
using DownMid = GemmShape<1, 4, 1, 1, 2, 6, 64>;    // 128 D cols x 64 tokens, 4 waves
// 65 to 96 tokens: one 96-token tile, which stages a quarter fewer rows of
// activations per weight tile than a 128-token tile (measured at D = 4096,
// F = 14336: T = 65, 80, 96 3.5-5% faster than the 128-token tiles; up to
// 64 tokens the 64-token tiles stay 8% faster).
using GateUpMid96 = GemmShape<2, 4, 1, 1, 3, 3, 64>; // 128 F cols x 96 tokens, 4 waves
using DownMid96 = GemmShape<1, 4, 1, 1, 3, 5, 64>;   // 128 D cols x 96 tokens, 4 waves
using DownMid160 = GemmShape<1, 4, 1, 1, 5, 3, 64>;  // 128 D cols x 160 tokens, 4 waves
using DownMid192 = GemmShape<1, 4, 1, 1, 6, 3, 64>;  // 128 D cols x 192 tokens, 4 waves
// The down steps of the one-launch MFMA kernel: the same tiles with 4 LDS
// stages, so that one LDS array per stage, shared with the gate/up step's,
// fits a CU (the ring depth does not change any sum: same bits).
using FusedDownTiny = GemmShape<1, 4, 1, 1, 1, 4, 64>;
using FusedDownMid = GemmShape<1, 4, 1, 1, 2, 4, 64>;
// The paired gate/up tiles (one weight per block, a G and a U block per
// column tile, EPI_GATE_PAIR) for one token tile of 65 to 192 tokens: the
// down step's tiles (with 3 stages at 128 tokens: 0.3 us faster than 4), and
// a 192-token tile.
using PairMid96 = GemmShape<1, 4, 1, 1, 3, 5, 64>; // 128 F cols x 96 tokens, 4 waves
using PairSmall = GemmShape<1, 2, 2, 2, 2, 3, 64>; // 128 F cols x 128 tokens, 4 waves
using PairMid160 = GemmShape<1, 4, 1, 1, 5, 3, 64>; // 128 F cols x 160 tokens, 4 waves
using PairMid192 = GemmShape<1, 4, 1, 1, 6, 3, 64>; // 128 F cols x 192 tokens, 4 waves
// 257 to 384 tokens: two 192-token tiles (a quarter less work and
// activation staging than two 256-token tiles at T = 384, a quarter more at
// T = 257 than needed instead of twice).
using GateUp192 = GemmShape<2, 4, 1, 1, 6, 4, 32>; // 128 F cols x 192 tokens, per weight, 4 waves
// Column tiles swept per token tile by consecutive blocks (L2 locality),
// from a sweep at T=4096/2048 on MI355X.
constexpr int kGroupGateUp = 8;
constexpr int kGroupDown = 8;

constexpr int kGemvMaxTokens = 8;
// The one-launch MFMA path (GMLP_PATH_FUSED_MFMA) runs the 32- and 64-token
// tiles: one token tile per step.
constexpr int kFusedMfmaMaxTokens = 64;
// The automatic path takes the GEMV kernels up to this many tokens.  From 6
// tokens the 32-token MFMA tiles are faster (measured at D = 4096,
// F = 14336 over rotated weights: 70.0-70.4 us against 72.5-73.7 us at
// T = 6, 70.2 against 75.4-76.4 at T = 7; the GEMV wins at T = 5, 64.7
// against 69.9), since a GEMV load batch shrinks to four rows from T = 3
// and to two from T = 7.
constexpr int kGemvAutoTokens = 5;
constexpr int64_t kMaxDim = int64_t(1) << 22; // D, F: keeps 32-bit tile offsets in range
// Tokens per call, and elements of any one tensor (2^37 bf16 = 256 GiB, more
// than one device holds).  Together they keep every tile count, block count
// and launch grid within int and within the 2^32 threads a launch
// dimension allows (the largest grid, 256-token tiles of 128 columns, has
// about T F / 32768 blocks of 512 threads).
constexpr int64_t kMaxTokens = int64_t(1) << 24;
constexpr int64_t kMaxElements = int64_t(1) << 37;

// Whether any of the [rows, a], [rows, b] and [a, b] tensors of a shape has
// more than kMaxElements elements (each factor already within its limit, so
// the products fit in int64).
bool too_many_elements(int64_t rows, int64_t a, int64_t b)
{
    return rows * a > kMaxElements || rows * b > kMaxElements || a * b > kMaxElements;
}
constexpr size_t kAlign = 256;
// Arrival counters sit at the start of every workspace in a block of fixed
// size (enough for any shape: at most kMaxDim / 256 GEMV strips, fewer than
// 256 split GEMM tiles), followed by the fused kernel's ready words (one
// 128-byte line per down split) and a line holding the fused kernel's
// give-up count, so a zeroed workspace stays valid when it is reused for
// another shape.  Every kernel leaves the counters and ready words zero; the
// give-up count stays until gmlp_workspace_status reads it.
constexpr size_t kStripCounterBytes = 64 * 1024;
constexpr int kCounterLine = 32; // words per 128-byte line
constexpr size_t kReadyBytes = (size_t)kFusedMaxSplits * kFlagStride * sizeof(uint32_t);
constexpr size_t kErrorOffset = kStripCounterBytes + kReadyBytes;
constexpr size_t kCounterBytes = kErrorOffset + 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

enum Kind {
    K_NONE,
    K_GEMM_GU_L, K_GEMM_GU_S, K_GEMM_GU_W, K_GEMM_GU_M, K_GEMM_GU_T, K_GEMM_GU_P, K_GEMM_GU_Y,
    K_GEMM_DN_L, K_GEMM_DN_S, K_GEMM_DN_W, K_GEMM_DN_M, K_GEMM_DN_T, K_GEMM_DN_X, K_GEMM_DN_Y, K_GEMM_DN_Q,
    K_GEMV
};

// One matmul step (gate/up or down) of a call.
struct Step {
    Kind kind = K_NONE;
    int M = 0, N = 0, K = 0;
    int tiles_m = 0, tiles_n = 0; // GEMM
    int group_m = 1;              // GEMM block order
    int strips = 0;               // GEMV
    int strip_lanes = 32;         // GEMV: 8-column lanes per row
    int counter_stride = 1;       // GEMV: words between two strips' arrival counters
    int splits = 1, k_split = 0;
    int blocks = 0, threads = 0;
    size_t partial_bytes = 0; // fp32 split-K partial sums
    int counters = 0;         // arrival counters
    // GEMM without split-K whose tiles leave a last round of blocks at most
    // half full: the first tile_count tiles (whole rounds) take one block
    // each, the last tail_tiles tail_splits blocks each over K (tail_k_split
    // rows each), so they fill a round instead of idling most of the chip;
    // both run as one split-K launch, the whole tiles' blocks first.
    int tile_base = 0, tile_count = 0;
    int tail_tiles = 0, tail_splits = 1, tail_k_split = 0;
    int64_t block_macs = 0; // GEMM: multiply-adds of one block of the main launch
};

// The split part of a step with a tail: its last tail_tiles tiles, split
// over K (launched after the step's tile_count whole-tile blocks).
Step tail_step(const Step &s)
{
    Step t = s;
    t.tile_base = s.tile_count;
    t.tile_count = s.tail_tiles;
    t.splits = s.tail_splits;
    t.k_split = s.tail_k_split;
    t.blocks = s.tail_tiles * s.tail_splits;
    t.tail_tiles = 0;
    return t;
}

struct Plan {
    int path = GMLP_PATH_AUTO;
    Step gate_up, down;
    // Gate/up on a token split: gate_up covers rows [0, rest_row), and
    // gate_up_rest, planned as a problem of its own, rows [rest_row, T).
    int64_t rest_row = 0;
    Step gate_up_rest;
};


struct Layout {
    size_t counters_off = 0, h_off = 0, partial_off = 0, rrms_off = 0, total = 0;
    int counters = 0; // most arrival counters any path uses for this shape
};

// Which member of the Gated MLP family a call computes.
struct Variant {
    int act = GMLP_ACT_SILU;
    float beta = 1.0f;
    bool rms = false; // RMSNorm in front
    float eps = 0.0f;
};

// Blocks of one round: one per CU of the MI355X (256 CUs).
constexpr int kBlockTarget = 256;
// Splits of a tail launch (see Step::tail_tiles).
constexpr int kMaxTailSplits = 8;
// Rows of K each split of a split-K large down tile keeps at least.
constexpr int kMinLargeSplitRows = 40 * DownLarge::BK;
// Large down tiles split into pieces shorter than this give way to the
// 256 x 128 tiles (64 k-tiles of 64 rows).
constexpr int kWideDownBelowRows = 64 * DownLarge::BK;

// Split K so that at most `target` blocks run (the small-T kernels hold one
// block per CU: a second round of blocks would cost a whole tile's time),
// keeping at least `min_tiles` k-tiles of `tile_k` rows per split.  Each
// split adds T x columns fp32 partial sums to write and read back, so the
// count rounds down.
void choose_splits(Step &s, int tiles, int target, int tile_k, int min_tiles)
{
    const int64_t ktiles = cdiv(s.K, tile_k);
    int64_t splits = 1;
    if (tiles < target)
        splits = std::min<int64_t>(target / tiles, std::max<int64_t>(1, ktiles / min_tiles));
    const int64_t per = cdiv(ktiles, splits);
    s.k_split = (int)(per * tile_k);
    s.splits = (int)cdiv(s.K, s.k_split);
}

template <class S>
void gemm_step(Step &s, Kind kind, int M, int N, int K, int nw, bool allow_split, int group_m)
{
    s.kind = kind;
    s.M = M;
    s.N = N;
    s.K = K;
    s.tiles_m = (int)cdiv(M, S::BMW);
    s.tiles_n = (int)cdiv(N, S::BN);
    s.group_m = std::max(1, std::min(group_m, s.tiles_m));
    const int tiles = s.tiles_m * s.tiles_n;
    s.tile_count = tiles;
    s.tail_tiles = 0;
    s.tail_splits = 1;
    s.tail_k_split = 0;
    if (allow_split)
        choose_splits(s, tiles, kBlockTarget, S::BK, 2);
    else {
        s.splits = 1;
        s.k_split = K;
        const int rem = tiles % kBlockTarget;
        if (tiles > kBlockTarget && rem > 0 && rem <= kBlockTarget / 2) {
            // At most 8 splits: the last block of a tile reads the other
            // splits' 256 x 256 partial tiles one after another.
            Step t = s;
            choose_splits(t, rem, std::min(kBlockTarget, kMaxTailSplits * rem), S::BK, 2);
            if (t.splits > 1) {
                s.tile_count = tiles - rem;
                s.tail_tiles = rem;
                s.tail_splits = t.splits;
                s.tail_k_split = t.k_split;
            }
        }
    }
    s.blocks = s.tile_count * s.splits;
    s.block_macs = (int64_t)S::BMW * S::BN * nw * s.k_split;
    s.threads = S::NTHREADS;
    s.counters = std::max(s.splits > 1 ? tiles : 0, s.tail_tiles);
    // Partial sums of whole tiles (padded), [split][tile][wave][piece][lane];
    // the tail tiles use the space of a split step's partial sums.
    const size_t tile_bytes = (size_t)S::BMW * S::BN * nw * sizeof(float);
    s.partial_bytes = std::max(s.splits > 1 ? (size_t)s.splits * tiles * tile_bytes : 0,
                               (size_t)s.tail_splits * s.tail_tiles * tile_bytes);
}

// The paired gate/up step (EPI_GATE_PAIR): one-weight tiles, a G and a U
// block per column tile, each over the whole of K.  It replaces a dual-B
// plan of one token tile that splits K in two (and, below, one of two
// 128-token tiles) where that plan's blocks fill more than three
// quarters of the chip: the same blocks and weight bytes, half the fp32
// exchange and 256-byte row segments of one weight per block, but each
// block stages all of X rather than half.  Measured at D = 4096 over
// rotated weights, gate/up alone (pairs against dual-B): 256 blocks
// (F = 16384) T = 100 53.1 against 57.8 us, T = 128 54.4 against 62.0; 224
// blocks (F = 14336) T = 65 48.9 against 51.3, T = 96 50.7-51.1 against
// 52.5-52.9, T = 128 53.8-54.7 against 54.6-56.0; 192 blocks (F = 12288)
// equal within 0.5%; 172 blocks (F = 11008) T = 100 47.1 against 45.1, where
// fewer CUs share the stream and the extra staging costs.  Up to 64 tokens
// (where the one-launch MFMA path runs the dual-B tiles) the gain is within
// 1-2%, so those keep the dual-B plan.
constexpr int kPairMinBlocks = kBlockTarget * 3 / 4 + 1;
template <class S>
void pair_step(Step &s, int M, int N, int K, int group_m)
{
    s.kind = K_GEMM_GU_P;
    s.M = M;
    s.N = N;
    s.K = K;
    s.tiles_m = (int)cdiv(M, S::BMW);
    s.tiles_n = (int)cdiv(N, S::BN);
    s.group_m = std::max(1, std::min(group_m, s.tiles_m));
    const int tiles = s.tiles_m * s.tiles_n;
    s.tile_count = tiles;
    s.tail_tiles = 0;
    s.tail_splits = 1;
    s.tail_k_split = 0;
    s.splits = 2; // the G and the U block of each tile
    s.k_split = K;
    s.blocks = 2 * tiles;
    s.threads = S::NTHREADS;
    s.counters = tiles;
    s.partial_bytes = (size_t)2 * tiles * S::BMW * S::BN * sizeof(float);
}

// Rows per load batch of all row groups of a block, per token count and
// step (splits are whole batches).
int gemv_batch_span(int nt, int nw)
{
    const int rg = gemv_threads(nt) / gemv_strip_lanes(nt, nw);
    auto rows = [nw](auto ntc) {
        constexpr int NT = decltype(ntc)::value;
        return nw == 2 ? gemv_batch_rows<NT, 2>() : gemv_batch_rows<NT, 1>();
    };
    switch (nt) {
    case 1: return rg * rows(std::integral_constant<int, 1>{});
    case 2: return rg * rows(std::integral_constant<int, 2>{});
    case 3: return rg * rows(std::integral_constant<int, 3>{});
    case 4: return rg * rows(std::integral_constant<int, 4>{});
    case 5: return rg * rows(std::integral_constant<int, 5>{});
    case 6: return rg * rows(std::integral_constant<int, 6>{});
    case 7: return rg * rows(std::integral_constant<int, 7>{});
    default: return rg * rows(std::integral_constant<int, 8>{});
    }
}

// GEMV decomposition: strips of 512 columns (64 lanes x 8: gate/up up to 4
// tokens) or 256 columns (32 lanes x 8) times k splits.  Measured on MI355X
// at D=4096, F=14336: one block per CU at most, as few splits as that
// allows, and splits of whole load batches are fastest (T = 1: gate/up 28
// strips x 8 splits of 512 rows, down 16 x 16 splits of 896 rows); more,
// shorter blocks add partial sums and reduction latency (down in 28 or 32
// splits: 2-4 us slower), and a second block on a CU does not raise its
// share of HBM bandwidth.
// For T = 7, 8 a load batch is only two rows (the accumulators of 8 tokens
// take the registers), so two 4-wave blocks per CU keep enough loads in
// flight (measured: T = 5, 6 are 9% and 4% faster with one block per CU,
// T = 7, 8 6% and 11% slower).
int gemv_block_target(int nt) { return nt <= 6 ? 256 : 512; }

void gemv_step(Step &s, int M, int N, int K, int nw)
{
    s.kind = K_GEMV;
    s.M = M;
    s.N = N;
    s.K = K;
    s.threads = gemv_threads(N);
    s.strip_lanes = gemv_strip_lanes(N, nw);
    s.strips = (int)cdiv(M, 8 * s.strip_lanes);
    const int span = gemv_batch_span(N, nw);
    const int64_t max_sp = std::max<int64_t>(1, std::min<int64_t>(gemv_block_target(N) / s.strips, cdiv(K, span)));
    int64_t rows = 0;
    for (int64_t sp = max_sp; sp >= 1 && !rows; --sp)
        if (K % sp == 0 && (K / sp) % span == 0)
            rows = K / sp; // equal splits of whole batches
    if (!rows || K / rows < max_sp / 2)
        rows = cdiv(cdiv(K, max_sp), span) * span; // nearly equal splits of whole batches
    s.k_split = (int)rows;
    s.splits = (int)cdiv(K, rows);
    s.blocks = s.strips * s.splits;
    s.counters = s.splits > 1 ? s.strips : 0;
    // Per-split column sums, then (gate/up with RMSNorm) per-strip, per-split
    // sums of squares of X.
    s.partial_bytes = s.splits > 1 ? (size_t)s.splits * ((size_t)nw * N * M + (size_t)s.strips * N) * sizeof(float) : 0;
}

Plan make_plan(int64_t T, int64_t D, int64_t F, int path)
{
    Plan p;
    const int asked = path;
    if (path == GMLP_PATH_AUTO)
        path = T <= kGemvAutoTokens ? GMLP_PATH_GEMV : GMLP_PATH_MFMA;
    p.path = path;
    if (path == GMLP_PATH_GEMV || path == GMLP_PATH_FUSED) {
        gemv_step(p.gate_up, (int)F, (int)T, (int)D, 2);
        gemv_step(p.down, (int)D, (int)T, (int)F, 1);
        // Each strip's arrival counter on a 128-byte line of its own where
        // both steps' counters fit so (the one-launch kernel holds them at
        // once): the arrivals of one strip's splits then do not queue behind
        // the other strips' atomics on a shared line.  Measured at the
        // decode shape (16 down strips of 16 splits): down step 21.3 ->
        // 20.3 us; the gate/up step (8 splits) unchanged.
        const int stride = (size_t)(p.gate_up.strips + p.down.strips) * kCounterLine * sizeof(uint32_t) <=
                                   kStripCounterBytes
                               ? kCounterLine
                               : 1;
        for (Step *s : {&p.gate_up, &p.down}) {
            s->counter_stride = stride;
            s->counters = s->splits > 1 ? s->strips * stride : 0;
        }
        return p;
    }
    if (path == GMLP_PATH_FUSED_MFMA) { // the few-token tiles whatever F and D are
        if (T <= GateUpTiny::BN) {
            gemm_step<GateUpTiny>(p.gate_up, K_GEMM_GU_T, (int)F, (int)T, (int)D, 2, true, kGroupGateUp);
            gemm_step<DownTiny>(p.down, K_GEMM_DN_T, (int)D, (int)T, (int)F, 1, true, kGroupDown);
        } else {
            gemm_step<GateUpMid>(p.gate_up, K_GEMM_GU_M, (int)F, (int)T, (int)D, 2, true, kGroupGateUp);
            gemm_step<DownMid>(p.down, K_GEMM_DN_M, (int)D, (int)T, (int)F, 1, true, kGroupDown);
        }
        return p;
    }
    // Gate/up: large tiles once there are enough of them to fill the chip,
    // and above 256 tokens once they at least nearly fill it: there one
    // round of large tiles beats the partial second round that small tiles
    // leave (measured at D = 4096, F = 14336: T = 320, 384 11% faster,
    // T = 512 and 1024 8%).
    const int64_t large_tiles = cdiv(T, GateUpLarge::BN) * cdiv(F, GateUpLarge::BMW);
    // Two 192-token tiles where they make one round that is at least three
    // quarters full (measured at D = 4096, F = 14336 against two 256-token
    // tiles, gate/up: T = 257 111.8 -> 89.0 us, 320 114.2 -> 93.5, 384
    // 115.8 -> 98.3; 8 waves with 64-row k-tiles were 6-11% slower).
    const int64_t tiles192 = cdiv(T, GateUp192::BN) * cdiv(F, GateUp192::BMW);
    if (T > 256 && T <= 2 * GateUp192::BN && tiles192 <= kBlockTarget && tiles192 >= kBlockTarget * 3 / 4)
        gemm_step<GateUp192>(p.gate_up, K_GEMM_GU_Y, (int)F, (int)T, (int)D, 2, false, kGroupGateUp);
    else if (large_tiles >= 512 || (T > 256 && large_tiles >= 192))
        gemm_step<GateUpLarge>(p.gate_up, K_GEMM_GU_L, (int)F, (int)T, (int)D, 2, false, kGroupGateUp);
    else if (T <= GateUpTiny::BN)
        gemm_step<GateUpTiny>(p.gate_up, K_GEMM_GU_T, (int)F, (int)T, (int)D, 2, true, kGroupGateUp);
    else if (T <= GateUpMid::BN)
        gemm_step<GateUpMid>(p.gate_up, K_GEMM_GU_M, (int)F, (int)T, (int)D, 2, true, kGroupGateUp);
    else if (T <= GateUpMid96::BN)
        gemm_step<GateUpMid96>(p.gate_up, K_GEMM_GU_W, (int)F, (int)T, (int)D, 2, true, kGroupGateUp);
    else
        gemm_step<GateUpSmall>(p.gate_up, K_GEMM_GU_S, (int)F, (int)T, (int)D, 2, true, kGroupGateUp);
    if ((p.gate_up.kind == K_GEMM_GU_W || p.gate_up.kind == K_GEMM_GU_S) && p.gate_up.tiles_n == 1 &&
        p.gate_up.splits == 2 && p.gate_up.blocks >= kPairMinBlocks) {
        if (T <= PairMid96::BN)
            pair_step<PairMid96>(p.gate_up, (int)F, (int)T, (int)D, kGroupGateUp);
        else
            pair_step<PairSmall>(p.gate_up, (int)F, (int)T, (int)D, kGroupGateUp);
    }
    // 129 to 192 tokens, where the dual-B plan runs two 128-token tiles
    // without split-K on as many blocks: one 192-token tile as pairs, each
    // weight element read once (the weights streamed) and X staged 1.5x
    // instead of twice per column tile.  Measured at D = 4096, F = 14336,
    // gate/up alone: T = 129 68.5 -> 67.4 us, 160 70.9 -> 68.4, 192 74.3 ->
    // 68.6-68.8; pairs of 256-token tiles for T = 193..256 were slower (T =
    // 224: 77.7 -> 89-91 us).  Up to 160 tokens a 160-token tile stages a
    // sixth less X and does a sixth less MFMA work: T = 129 67.9 -> 58.3
    // us, 144 69.4 -> 58.6, 160 69.0 -> 59.3.
    if (p.gate_up.kind == K_GEMM_GU_S && p.gate_up.tiles_n == 2 && p.gate_up.splits == 1 && T <= PairMid192::BN &&
        p.gate_up.blocks >= kPairMinBlocks && p.gate_up.blocks <= kBlockTarget) {
        if (T <= PairMid160::BN)
            pair_step<PairMid160>(p.gate_up, (int)F, (int)T, (int)D, kGroupGateUp);
        else
            pair_step<PairMid192>(p.gate_up, (int)F, (int)T, (int)D, kGroupGateUp);
    }
    // Down: large tiles once there are enough of them to fill the chip.
    // Above one token tile, from 40 of them up to a round, large tiles split over K to fill one
    // round beat two rounds of 128 x 128 tiles (measured: D = 4096, F = 14336
    // at T = 640 and 2048 6-8% faster, T = 1024 equal; D = 8192, F = 28672 at
    // T = 512..1280 6-15% faster), while each split keeps at least 40
    // k-tiles (D = 2048, F = 8192 at T = 2048, 4 splits of 32 k-tiles: 10%
    // slower).
    const int64_t down_large = cdiv(T, DownLarge::BN) * cdiv(D, DownLarge::BMW);
    Step large_down;
    if (T > DownLarge::BN && down_large >= 40 && down_large < 192)
        gemm_step<DownLarge>(large_down, K_GEMM_DN_L, (int)D, (int)T, (int)F, 1, true, kGroupDown);
    // Where the large tiles' splits would be shorter than 64 k-tiles, and
    // above 256 tokens where they are not used at all, 256 x 128 tiles split
    // over K in splits of at least 40 k-tiles (measured at D = 4096,
    // F = 14336: down step 6-24% faster at T = 257..1024, the step 2-10%;
    // D = 8192, F = 28672, whose large-tile splits are 7168 rows and more,
    // keep the large tiles; T = 300, D = 1032, F = 2056 would split 11 ways
    // into 187-row pieces: 45% slower, so excluded by the minimum).
    Step wide;
    if (T > 256 && down_large < 192)
        gemm_step<DownWide>(wide, K_GEMM_DN_X, (int)D, (int)T, (int)F, 1, true, kGroupDown);
    const bool large_ok =
        large_down.kind == K_GEMM_DN_L && (large_down.splits == 1 || large_down.k_split >= kMinLargeSplitRows);
    const bool wide_ok = wide.kind == K_GEMM_DN_X && wide.splits >= 2 && wide.k_split >= kMinLargeSplitRows &&
                         (!large_ok || large_down.k_split < kWideDownBelowRows);
    if (down_large >= 192)
        gemm_step<DownLarge>(p.down, K_GEMM_DN_L, (int)D, (int)T, (int)F, 1, false, kGroupDown);
    else if (wide_ok)
        p.down = wide;
    else if (large_ok)
        p.down = large_down;
    else if (T <= DownTiny::BN)
        gemm_step<DownTiny>(p.down, K_GEMM_DN_T, (int)D, (int)T, (int)F, 1, true, kGroupDown);
    else if (T <= DownMid::BN)
        gemm_step<DownMid>(p.down, K_GEMM_DN_M, (int)D, (int)T, (int)F, 1, true, kGroupDown);
    else if (T <= DownMid96::BN)
        gemm_step<DownMid96>(p.down, K_GEMM_DN_W, (int)D, (int)T, (int)F, 1, true, kGroupDown);
    // 129 to 192 tokens: one 192-token tile split over K instead of two
    // 128-token tiles, so each weight element is read once (measured:
    // steps at D = 4096, F = 14336 T = 129 109.6 -> 108.8 us, 160 112.1 ->
    // 110.1, 192 115.4 -> 111.2; D = 8192, F = 28672 T = 160 454.8 -> 412.9).
    // Up to 160 tokens a 160-token tile (down at D = 8192, F = 28672: T =
    // 129 108.2-109.6 -> 98.0-98.5 us, 150 111.4 -> 100.4; equal at
    // D = 4096, F = 14336).
    else if (T > DownSmall::BN && T <= DownMid160::BN)
        gemm_step<DownMid160>(p.down, K_GEMM_DN_Q, (int)D, (int)T, (int)F, 1, true, kGroupDown);
    else if (T > DownSmall::BN && T <= DownMid192::BN)
        gemm_step<DownMid192>(p.down, K_GEMM_DN_Y, (int)D, (int)T, (int)F, 1, true, kGroupDown);
    else
        gemm_step<DownSmall>(p.down, K_GEMM_DN_S, (int)D, (int)T, (int)F, 1, true, kGroupDown);
    // 257 to 384 tokens: two 192-token down tiles split over K where there
    // are 64 to 128 of them (so that at least two splits fill a round) and
    // a block's work is at most 95% of what the rules above give it.
    // Measured: down at D = 4096, F = 14336 T = 257 61.9 -> 58.7 us, 320
    // 62.4 -> 59.9, 384 62.9 -> 60.4 (93% of the work); D = 8192, F = 28672,
    // T = 320 221.9 -> 195.0 (75%); slower at equal work (D = 5120,
    // F = 13824, T = 300: 69.5 -> 74.7) and with 32 tiles (D = 2048,
    // F = 8192, T = 300: 27.5 -> 34.4).
    const int64_t down192 = cdiv(T, DownMid192::BN) * cdiv(D, DownMid192::BMW);
    if (T > 256 && T <= 2 * DownMid192::BN && down192 >= 64 && down192 <= kBlockTarget / 2) {
        Step mid;
        gemm_step<DownMid192>(mid, K_GEMM_DN_Y, (int)D, (int)T, (int)F, 1, true, kGroupDown);
        if (p.down.tail_tiles == 0 && p.down.blocks <= kBlockTarget && mid.block_macs * 20 <= p.down.block_macs * 19)
            p.down = mid;
    }
    // From 513 tokens, where the 256-token gate/up tiles leave a last round
    // of split-K tail tiles and the last token tile is at most half full,
    // its r tokens may run as a gate/up problem of their own after the
    // whole 256-token tiles (few-token tiles that stream the weights,
    // mostly from the last-level cache) instead of padding them to 256
    // tokens.  The choice follows a cost in rounds of full-K tiles fitted
    // to measurements: a partial round costs a round, tail tiles split s
    // ways 1/s + 0.27, the r-token problem 0.9 C / 256 for C column tiles
    // (it streams weights that a round of tiles reads in about 280 tiles'
    // time).  Gate/up at D = 4096, F = 14336: T = 520 176.0 -> 148.9 us,
    // 640 178.0 -> 155.6, 1088 277.0 -> 252.5, 1600 364.8 -> 347.1, 2340
    // 490.2 -> 467.0, 2880 578.0 -> 562.8, kept whole at 1800 (388.7, split
    // 407.4); at D = 8192, F = 28672: T = 1100 1004.9 -> 932.5, 1600 1380.4
    // -> 1329.3, kept whole at 800 (762.2, split 797.6).  The down step
    // keeps one plan: splitting it was slower at every measured T.
    const int64_t rest = T % GateUpLarge::BN;
    if (p.gate_up.kind == K_GEMM_GU_L && rest > 0 && rest <= GateUpLarge::BN / 2 && T > 2 * GateUpLarge::BN) {
        const auto rounds_milli = [](const Step &s) {
            const int64_t full = s.tile_count / kBlockTarget, part = s.tile_count % kBlockTarget;
            return 1000 * (full + (part ? 1 : 0)) + (s.tail_tiles ? 1000 / s.tail_splits + 270 : 0);
        };
        const Step head = make_plan(T - rest, D, F, asked).gate_up;
        const int64_t rest_milli = 900 * (int64_t)p.gate_up.tiles_m / kBlockTarget;
        if (head.kind == K_GEMM_GU_L && rounds_milli(head) + rest_milli < rounds_milli(p.gate_up)) {
            p.gate_up = head;
            p.gate_up_rest = make_plan(rest, D, F, asked).gate_up;
            p.rest_row = T - rest;
        }
    }
    return p;
}

// Whether both steps' split-K counters of a one-launch MFMA plan fit in the
// counter block together (down's follow gate/up's).
bool fused_mfma_counters_fit(const Plan &p)
{
    return (size_t)(p.gate_up.tile_count + p.down.counters) * sizeof(uint32_t) <= kStripCounterBytes;
}

// One layout serves every path, so a workspace sized by gmlp_workspace_size
// fits whichever kernels run.
Layout make_layout(int64_t T, int64_t D, int64_t F)
{
    // T = 0 launches nothing; its workspace is sized as for one token (the
    // plans below need at least one token tile).
    T = std::max<int64_t>(T, 1);
    int counters = 0;
    size_t partial = 0;
    for (int path : {GMLP_PATH_GEMV, GMLP_PATH_MFMA}) {
        if (path == GMLP_PATH_GEMV && T > kGemvMaxTokens)
            continue;
        const Plan p = make_plan(T, D, F, path);
        counters = std::max({counters, p.gate_up.counters, p.down.counters, p.gate_up_rest.counters});
        partial = std::max({partial, p.gate_up.partial_bytes, p.down.partial_bytes, p.gate_up_rest.partial_bytes});
        if (path == GMLP_PATH_GEMV) // the fused kernel runs both steps at once: separate partial sums
            partial = std::max(partial, align_up(p.gate_up.partial_bytes) + p.down.partial_bytes);
    }
    if (T <= kFusedMfmaMaxTokens) {
        // The one-launch MFMA path: both steps' partial sums and counters at
        // once (where its counters fit the block: otherwise the path refuses
        // the shape and the other paths keep their workspace).
        const Plan p = make_plan(T, D, F, GMLP_PATH_FUSED_MFMA);
        if (fused_mfma_counters_fit(p)) {
            counters = std::max(counters, p.gate_up.tile_count + p.down.counters);
            partial = std::max(partial, align_up(p.gate_up.partial_bytes) + p.down.partial_bytes);
        }
    }
    Layout l;
    l.counters_off = 0;
    l.h_off = kCounterBytes;
    l.counters = counters;
    l.partial_off = l.h_off + align_up((size_t)T * F * 2);
    l.rrms_off = l.partial_off + align_up(partial);
    l.total = l.rrms_off + align_up((size_t)T * sizeof(float));
    return l;
}

bool misaligned(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) != 0; }

bool overlaps(const void *a, size_t an, const void *b, size_t bn)
{
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return an && bn && x < y + bn && y < x + an;
}

int check_shape(int64_t T, int64_t D, int64_t F)
{
    if (T < 0 || D <= 0 || F <= 0)
        return fail(GMLP_ERR_INVALID_ARG, "invalid shape T=%lld D=%lld F=%lld (need T >= 0, D > 0, F > 0)",
                    (long long)T, (long long)D, (long long)F);
    if (D % 8 || F % 8)
        return fail(GMLP_ERR_UNSUPPORTED, "D=%lld and F=%lld must be multiples of 8", (long long)D,
                    (long long)F);
    if (D > kMaxDim || F > kMaxDim || T > kMaxTokens || too_many_elements(T, D, F))
        return fail(GMLP_ERR_UNSUPPORTED, "shape T=%lld D=%lld F=%lld exceeds the supported range "
                    "(D, F <= %lld, T <= %lld, at most %lld elements per tensor)", (long long)T, (long long)D,
                    (long long)F, (long long)kMaxDim, (long long)kMaxTokens, (long long)kMaxElements);
    return GMLP_OK;
}

int check_ptr(const void *p, const char *name, bool required)
{
    if (!p)
        return required ? fail(GMLP_ERR_INVALID_ARG, "%s is NULL", name) : GMLP_OK;
    if (misaligned(p))
        return fail(GMLP_ERR_UNSUPPORTED, "%s (%p) is not 16-byte aligned", name, p);
    return GMLP_OK;
}

int validate(int64_t T, int64_t D, int64_t F, const void *X, const void *Wg, const void *Wu,
             const void *Wd, const void *Y)
{
    int rc;
    if ((rc = check_shape(T, D, F)))
        return rc;
    const bool rows = T > 0;
    if ((rc = check_ptr(X, "X", rows)) || (rc = check_ptr(Wg, "Wg", true)) ||
        (rc = check_ptr(Wu, "Wu", true)) || (rc = check_ptr(Wd, "Wd", true)) ||
        (rc = check_ptr(Y, "Y", rows)))
        return rc;
    const size_t xb = (size_t)T * D * 2, wb = (size_t)D * F * 2;
    if (overlaps(Y, xb, X, xb) || overlaps(Y, xb, Wg, wb) || overlaps(Y, xb, Wu, wb) ||
        overlaps(Y, xb, Wd, wb))
        return fail(GMLP_ERR_INVALID_ARG, "Y overlaps an input");
    return GMLP_OK;
}

// Weights are streamed (nontemporal loads) when the plan has a single token
// tile: then each weight element is read by one block only.
bool stream_weights(const Step &s) { return s.tiles_n == 1; }

// The fused kernel: the gate/up items on the first blocks, the down items on
// the rest, all in one launch.
int fused_grid(const Plan &plan) { return plan.gate_up.blocks + plan.down.blocks; }

int check_variant(int activation, float beta, int rmsnorm, float eps, Variant *v)
{
    if (activation != GMLP_ACT_SILU && activation != GMLP_ACT_SWISH && activation != GMLP_ACT_SIGMOID)
        return fail(GMLP_ERR_INVALID_ARG, "unknown activation %d", activation);
    if (!std::isfinite(beta))
        return fail(GMLP_ERR_INVALID_ARG, "beta must be finite");
    if (rmsnorm != 0 && rmsnorm != 1)
        return fail(GMLP_ERR_INVALID_ARG, "rmsnorm must be 0 or 1 (got %d)", rmsnorm);
    if (rmsnorm && !(std::isfinite(eps) && eps >= 0.0f))
        return fail(GMLP_ERR_INVALID_ARG, "eps must be finite and >= 0");
    v->act = activation;
    v->beta = activation == GMLP_ACT_SWISH ? beta : 1.0f;
    v->rms = rmsnorm != 0;
    v->eps = rmsnorm ? eps : 0.0f;
    return GMLP_OK;
}

int check_path(int path, int64_t T)
{
    if (path != GMLP_PATH_AUTO && path != GMLP_PATH_GEMV && path != GMLP_PATH_MFMA && path != GMLP_PATH_FUSED &&
        path != GMLP_PATH_FUSED_MFMA)
        return fail(GMLP_ERR_INVALID_ARG, "unknown path %d", path);
    if ((path == GMLP_PATH_GEMV || path == GMLP_PATH_FUSED) && T > kGemvMaxTokens)
        return fail(GMLP_ERR_UNSUPPORTED, "%s path needs T <= %d (T=%lld)",
                    path == GMLP_PATH_GEMV ? "GEMV" : "fused", kGemvMaxTokens, (long long)T);
    if (path == GMLP_PATH_FUSED_MFMA && T > kFusedMfmaMaxTokens)
        return fail(GMLP_ERR_UNSUPPORTED, "fused MFMA path needs T <= %d (T=%lld)", kFusedMfmaMaxTokens,
                    (long long)T);
    return GMLP_OK;
}

// The entry points that run one step alone (and Softmax+MatMul) have no
// fused form.
int check_single_step_path(int path, int64_t T)
{
    if (path == GMLP_PATH_FUSED || path == GMLP_PATH_FUSED_MFMA)
        return fail(GMLP_ERR_UNSUPPORTED, "the fused paths run the whole Gated MLP only");
    return check_path(path, T);
}

int check_workspace(void *ws, size_t ws_bytes, const Layout &l)
{
    if (!ws)
        return fail(GMLP_ERR_INVALID_ARG, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(ws) % kAlign)
        return fail(GMLP_ERR_UNSUPPORTED, "workspace %p is not %zu-byte aligned", ws, kAlign);
    if (ws_bytes < l.total)
        return fail(GMLP_ERR_NO_MEMORY, "workspace of %zu bytes, %zu needed", ws_bytes, l.total);
    if ((size_t)l.counters * sizeof(uint32_t) > kStripCounterBytes)
        return fail(GMLP_ERR_UNSUPPORTED, "shape needs %d arrival counters, more than the %zu reserved",
                    l.counters, kCounterBytes / sizeof(uint32_t));
    return GMLP_OK;
}

template <class S>
std::string shape_name()
{
    return "GemmShape<" + std::to_string(S::NW) + ", " + std::to_string(S::WM) + ", " +
           std::to_string(S::WN) + ", " + std::to_string(S::TM) + ", " + std::to_string(S::TN) + ", " +
           std::to_string(S::STAGES) + ", " + std::to_string(S::BK) + ">";
}

// A step's kernel as a profiler names it, without the namespace.
std::string kernel_name(const Step &s, bool gate_up)
{
    switch (s.kind) {
    case K_GEMM_GU_L: return "gemm_mfma_kernel<" + shape_name<GateUpLarge>() + ", 0, false, false>";
    case K_GEMM_GU_S:
        return "gemm_mfma_kernel<" + shape_name<GateUpSmall>() + ", 0, true, " + (stream_weights(s) ? "true>" : "false>");
    case K_GEMM_DN_L:
        return "gemm_mfma_kernel<" + shape_name<DownLarge>() + (s.splits > 1 ? ", 1, true, false>" : ", 1, false, false>");
    case K_GEMM_DN_X: return "gemm_mfma_kernel<" + shape_name<DownWide>() + ", 1, true, false>";
    case K_GEMM_DN_S:
        return "gemm_mfma_kernel<" + shape_name<DownSmall>() + ", 1, true, " + (stream_weights(s) ? "true>" : "false>");
    case K_GEMM_GU_T: return "gemm_mfma_kernel<" + shape_name<GateUpTiny>() + ", 0, true, true>";
    case K_GEMM_DN_T: return "gemm_mfma_kernel<" + shape_name<DownTiny>() + ", 1, true, true>";
    case K_GEMM_GU_M:
        return "gemm_mfma_kernel<" + shape_name<GateUpMid>() + ", 0, true, " + (stream_weights(s) ? "true>" : "false>");
    case K_GEMM_DN_M:
        return "gemm_mfma_kernel<" + shape_name<DownMid>() + ", 1, true, " + (stream_weights(s) ? "true>" : "false>");
    case K_GEMM_GU_W: return "gemm_mfma_kernel<" + shape_name<GateUpMid96>() + ", 0, true, true>";
    case K_GEMM_GU_Y: return "gemm_mfma_kernel<" + shape_name<GateUp192>() + ", 0, false, false>";
    case K_GEMM_DN_W: return "gemm_mfma_kernel<" + shape_name<DownMid96>() + ", 1, true, true>";
    case K_GEMM_DN_Q: return "gemm_mfma_kernel<" + shape_name<DownMid160>() + ", 1, true, true>";
    case K_GEMM_DN_Y:
        return "gemm_mfma_kernel<" + shape_name<DownMid192>() + ", 1, true, " + (stream_weights(s) ? "true>" : "false>");
    case K_GEMM_GU_P: {
        const std::string shape = s.N <= PairMid96::BN   ? shape_name<PairMid96>()
                                  : s.N <= PairSmall::BN ? shape_name<PairSmall>()
                                  : s.N <= PairMid160::BN ? shape_name<PairMid160>()
                                                         : shape_name<PairMid192>();
        return "gemm_mfma_kernel<" + shape + ", 2, true, true>";
    }
    case K_GEMV:
        return "gemv_splitk_kernel<" + std::to_string(s.N) + (gate_up ? ", 2, 0, false>" : ", 1, 1, false>");
    default: return "none";
    }
}

// The kernel of a fused plan as a profiler names it, without the namespace.
std::string fused_kernel_name(const Plan &plan)
{
    if (plan.path == GMLP_PATH_FUSED)
        return "gemv_fused_kernel<" + std::to_string(plan.gate_up.N) + ", false>";
    if (plan.gate_up.kind == K_GEMM_GU_T)
        return "gemm_fused_kernel<" + shape_name<GateUpTiny>() + ", " + shape_name<FusedDownTiny>() + ">";
    return "gemm_fused_kernel<" + shape_name<GateUpMid>() + ", " + shape_name<FusedDownMid>() + ">";
}

// The describe line of a step's launch.
std::string describe_step(const Step &s, bool gate_up)
{
    char tmp[200];
    if (s.tail_tiles) {
        // One split-K launch: the whole tiles first, one block each over
        // all of K, then the tail tiles' splits.
        const Step t = tail_step(s);
        const std::string shape = s.kind == K_GEMM_GU_L ? shape_name<GateUpLarge>() + ", 0" : shape_name<DownLarge>() + ", 1";
        snprintf(tmp, sizeof tmp, "gemm_mfma_kernel<%s, true, false> grid=%d block=%d k_splits=%d\n", shape.c_str(),
                 s.tile_count + t.blocks, t.threads, t.splits);
        return tmp;
    }
    snprintf(tmp, sizeof tmp, "%s grid=%d block=%d k_splits=%d\n", kernel_name(s, gate_up).c_str(), s.blocks,
             s.threads, s.splits);
    return tmp;
}

int check_gate_up_args(const void *X, const void *Wg, const void *Wu, const void *H, int64_t T,
                       int64_t D, int64_t F)
{
    int rc;
    if ((rc = check_shape(T, D, F)) || (rc = check_ptr(X, "X", T > 0)) ||
        (rc = check_ptr(Wg, "Wg", true)) || (rc = check_ptr(Wu, "Wu", true)) ||
        (rc = check_ptr(H, "H", T > 0)))
        return rc;
    const size_t hb = (size_t)T * F * 2, xb = (size_t)T * D * 2, wb = (size_t)D * F * 2;
    if (overlaps(H, hb, X, xb) || overlaps(H, hb, Wg, wb) || overlaps(H, hb, Wu, wb))
        return fail(GMLP_ERR_INVALID_ARG, "H overlaps an input");
    return GMLP_OK;
}

int check_down_args(const void *H, const void *Wd, const void *Y, int64_t T, int64_t F, int64_t D)
{
    int rc;
    if ((rc = check_shape(T, D, F)) || (rc = check_ptr(H, "H", T > 0)) ||
        (rc = check_ptr(Wd, "Wd", true)) || (rc = check_ptr(Y, "Y", T > 0)))
        return rc;
    const size_t hb = (size_t)T * F * 2, yb = (size_t)T * D * 2, wb = (size_t)D * F * 2;
    if (overlaps(Y, yb, H, hb) || overlaps(Y, yb, Wd, wb))
        return fail(GMLP_ERR_INVALID_ARG, "Y overlaps an input");
    return GMLP_OK;
}


int check_smm_shape(int64_t M, int64_t K, int64_t N)
{
    if (M < 0 || K <= 0 || N <= 0)
        return fail(GMLP_ERR_INVALID_ARG, "invalid shape M=%lld K=%lld N=%lld (need M >= 0, K > 0, N > 0)",
                    (long long)M, (long long)K, (long long)N);
    if (K % 8 || N % 8)
        return fail(GMLP_ERR_UNSUPPORTED, "K=%lld and N=%lld must be multiples of 8", (long long)K,
                    (long long)N);
    if (K > kMaxDim || N > kMaxDim || M > kMaxTokens || too_many_elements(M, K, N))
        return fail(GMLP_ERR_UNSUPPORTED, "shape M=%lld K=%lld N=%lld exceeds the supported range "
                    "(K, N <= %lld, M <= %lld, at most %lld elements per tensor)", (long long)M, (long long)K,
                    (long long)N, (long long)kMaxDim, (long long)kMaxTokens, (long long)kMaxElements);
    return GMLP_OK;
}

int check_smm_args(const void *X, const void *Y, const void *Z, int64_t M, int64_t K, int64_t N)
{
    int rc;
    if ((rc = check_smm_shape(M, K, N)))
        return rc;
    if ((rc = check_ptr(X, "X", M > 0)) || (rc = check_ptr(Y, "Y", true)) || (rc = check_ptr(Z, "Z", M > 0)))
        return rc;
    const size_t xb = (size_t)M * K * 2, yb = (size_t)K * N * 2, zb = (size_t)M * N * 2;
    if (overlaps(Z, zb, X, xb) || overlaps(Z, zb, Y, yb))
        return fail(GMLP_ERR_INVALID_ARG, "Z overlaps an input");
    return GMLP_OK;
}

// The automatic path keeps the GEMV kernel up to 8 rows here: at the square
// shapes of the benchmark (K = N = 8192) it beats the 32-token MFMA tiles at
// every M <= 8 (measured: 33.0 against 34.2 us at M = 8), unlike the
// Gated MLP's pair of steps.
Step smm_matmul_step(int64_t M, int64_t K, int64_t N, int path)
{
    if (path == GMLP_PATH_AUTO)
        path = M <= kGemvMaxTokens ? GMLP_PATH_GEMV : GMLP_PATH_MFMA;
    return make_plan(M, N, K, path).down;
}

// Counter block, then P [M, K] bf16 (in the H slot), the matmul's split-K
// partial sums, and the row sums [M] fp32 (in the row-scale slot).  Sized for
// every path of the shape.
Layout smm_layout(int64_t M, int64_t K, int64_t N)
{
    M = std::max<int64_t>(M, 1); // as for make_layout: M = 0 launches nothing
    int counters = 0;
    size_t partial = 0;
    for (int path : {GMLP_PATH_GEMV, GMLP_PATH_MFMA}) {
        if (path == GMLP_PATH_GEMV && M > kGemvMaxTokens)
            continue;
        const Step s = smm_matmul_step(M, K, N, path);
        counters = std::max(counters, s.counters);
        partial = std::max(partial, s.partial_bytes);
    }
    Layout l;
    l.counters_off = 0;
    l.counters = counters;
    l.h_off = kCounterBytes;
    l.partial_off = l.h_off + align_up((size_t)M * K * 2);
    l.rrms_off = l.partial_off + align_up(partial);
    l.total = l.rrms_off + align_up((size_t)M * sizeof(float));
    return l;
}

} // namespace
} // namespace gmlp
