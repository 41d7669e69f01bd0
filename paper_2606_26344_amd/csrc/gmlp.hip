// libgmlp.so: the C ABI of include/gmlp.h (the Gated MLP family) and
// include/softmax_matmul.h (Softmax+MatMul) on top of the gfx950 kernels.
//
// Host side only: argument validation, the choice of kernels and tile
// configuration for a shape (the library's static analogue of the paper's
// empirical per-shape selection, Section 4.6), workspace layout and launches.
// Every arithmetic step runs in the kernels of gemm_mfma.hpp, gemv.hpp,
// rmsnorm.hpp and softmax.hpp.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cmath>
#include <cstring>
#include <atomic>
#include <mutex>
#include <string>

#include "gmlp.h"
#include "softmax_matmul.h"
#include "gemm_mfma.hpp"
#include "gemv.hpp"
#include "rmsnorm.hpp"
#include "softmax.hpp"

using namespace gmlp;

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
using GateUpLarge = GemmShape<2, 4, 2, 1, 4, 3, 32>; // 128 F cols x 256 tokens, per weight, 8 waves
using GateUpSmall = GemmShape<2, 4, 2, 1, 2, 3, 64>; // 128 F cols x 128 tokens, 8 waves
using DownLarge = GemmShape<1, 4, 2, 2, 4, 2, 64>;   // 256 D cols x 256 tokens, 8 waves
using DownSmall = GemmShape<1, 2, 2, 2, 2, 4, 64>;   // 128 D cols x 128 tokens
// Up to 32 tokens: the same weight tiles with one 32-token tile, so the
// activations staged per weight byte drop fourfold.
using GateUpTiny = GemmShape<2, 4, 1, 1, 1, 4, 64>; // 128 F cols x 32 tokens, 4 waves
using DownTiny = GemmShape<1, 4, 1, 1, 1, 6, 64>;   // 128 D cols x 32 tokens, 4 waves
using GateUpMid = GemmShape<2, 4, 1, 1, 2, 3, 64>;  // 128 F cols x 64 tokens, 4 waves
using DownMid = GemmShape<1, 4, 1, 1, 2, 6, 64>;    // 128 D cols x 64 tokens, 4 waves
// Column tiles swept per token tile by consecutive blocks (L2 locality),
// from a sweep at T=4096/2048 on MI355X.
constexpr int kGroupGateUp = 8;
constexpr int kGroupDown = 8;

constexpr int kGemvMaxTokens = 8;
// The automatic path takes the GEMV kernels up to this many tokens.  From 7
// tokens the 32-token MFMA tiles are faster (measured at D = 4096,
// F = 14336: 70.7 us against 74.6 us at T = 7 and 76.7 us at T = 8; equal at
// T = 6), since a GEMV load batch shrinks to two rows there.
constexpr int kGemvAutoTokens = 6;
constexpr int64_t kMaxDim = int64_t(1) << 22; // D, F: keeps 32-bit tile offsets in range
constexpr int64_t kMaxTokens = int64_t(1) << 30;
constexpr size_t kAlign = 256;
// Arrival counters sit at the start of every workspace in a block of fixed
// size (enough for any shape: at most kMaxDim / 256 GEMV strips, fewer than
// 256 split GEMM tiles), followed by the fused kernel's ready words (one
// 128-byte line per down split) and a line holding the fused kernel's
// give-up count, so a zeroed workspace stays valid when it is reused for
// another shape.  Every kernel leaves the counters and ready words zero; the
// give-up count stays until gmlp_workspace_status reads it.
constexpr size_t kStripCounterBytes = 64 * 1024;
constexpr size_t kReadyBytes = (size_t)kFusedMaxSplits * kFlagStride * sizeof(uint32_t);
constexpr size_t kErrorOffset = kStripCounterBytes + kReadyBytes;
constexpr size_t kCounterBytes = kErrorOffset + 256;
// Polls of a ready word (each with a short sleep) before a down block of the
// fused kernel stops waiting: about a second, far beyond any real wait.
// gmlp_test_fused_spin_limit changes it (tests force a give-up with 0).
constexpr uint32_t kSpinLimit = 1u << 20;
std::atomic<uint32_t> g_spin_limit{kSpinLimit};

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

enum Kind { K_NONE, K_GEMM_GU_L, K_GEMM_GU_S, K_GEMM_GU_M, K_GEMM_GU_T, K_GEMM_DN_L, K_GEMM_DN_S, K_GEMM_DN_M, K_GEMM_DN_T, K_GEMV };

// One matmul step (gate/up or down) of a call.
struct Step {
    Kind kind = K_NONE;
    int M = 0, N = 0, K = 0;
    int tiles_m = 0, tiles_n = 0; // GEMM
    int group_m = 1;              // GEMM block order
    int strips = 0;               // GEMV
    int strip_lanes = 32;         // GEMV: 8-column lanes per row
    int splits = 1, k_split = 0;
    int blocks = 0, threads = 0;
    size_t partial_bytes = 0; // fp32 split-K partial sums
    int counters = 0;         // arrival counters
    // GEMM without split-K whose tiles leave a last round of blocks at most
    // half full: the first tile_count tiles (whole rounds) run as planned,
    // the last tail_tiles run in a second launch split tail_splits ways over
    // K (tail_k_split rows each), so they fill a round instead of idling most
    // of the chip.
    int tile_base = 0, tile_count = 0;
    int tail_tiles = 0, tail_splits = 1, tail_k_split = 0;
};

// The second launch of a step with a tail: its last tail_tiles tiles, split
// over K.
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
    s.threads = S::NTHREADS;
    s.counters = std::max(s.splits > 1 ? tiles : 0, s.tail_tiles);
    // Partial sums of whole tiles (padded), [split][tile][wave][piece][lane];
    // the tail launch runs after the main one and reuses the space.
    const size_t tile_bytes = (size_t)S::BMW * S::BN * nw * sizeof(float);
    s.partial_bytes = std::max(s.splits > 1 ? (size_t)s.splits * tiles * tile_bytes : 0,
                               (size_t)s.tail_splits * s.tail_tiles * tile_bytes);
}

// Rows per load batch of the 8 row groups, per token count (splits are
// whole batches).
int gemv_batch_span(int nt)
{
    switch (nt) {
    case 1: return 8 * gemv_batch_rows<1>();
    case 2: return 8 * gemv_batch_rows<2>();
    case 3: return 8 * gemv_batch_rows<3>();
    case 4: return 8 * gemv_batch_rows<4>();
    case 5: return 8 * gemv_batch_rows<5>();
    case 6: return 8 * gemv_batch_rows<6>();
    case 7: return 8 * gemv_batch_rows<7>();
    default: return 8 * gemv_batch_rows<8>();
    }
}

// GEMV decomposition: strips of 256 columns (32 lanes x 8) times k splits.
// Measured on MI355X at D=4096, F=14336 (T=1): one block per CU at most, as
// few splits as that allows, and splits of whole load batches are fastest
// (gate/up 56 strips x 4 splits, down 16 x 14: 224 blocks of 1024 rows);
// more, shorter blocks add partial sums and reduction latency, and a second
// block on a CU does not raise its share of HBM bandwidth.
// For T = 7, 8 a load batch is only two rows (the accumulators of 8 tokens
// take the registers), so two blocks per CU keep enough loads in flight
// (measured: T = 5, 6 are 9% and 4% faster with one block per CU, T = 7, 8
// 6% and 11% slower).
int gemv_block_target(int nt) { return nt <= 6 ? 256 : 512; }

void gemv_step(Step &s, int M, int N, int K, int nw)
{
    s.kind = K_GEMV;
    s.M = M;
    s.N = N;
    s.K = K;
    s.threads = kGemvThreads;
    s.strip_lanes = 32;
    s.strips = (int)cdiv(M, 8 * s.strip_lanes);
    const int span = gemv_batch_span(N);
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
    if (path == GMLP_PATH_AUTO)
        path = T <= kGemvAutoTokens ? GMLP_PATH_GEMV : GMLP_PATH_MFMA;
    p.path = path;
    if (path == GMLP_PATH_GEMV || path == GMLP_PATH_FUSED) {
        gemv_step(p.gate_up, (int)F, (int)T, (int)D, 2);
        gemv_step(p.down, (int)D, (int)T, (int)F, 1);
        return p;
    }
    // Gate/up: large tiles once there are enough of them to fill the chip,
    // and above 256 tokens once they at least nearly fill it: there one
    // round of large tiles beats the partial second round that small tiles
    // leave (measured at D = 4096, F = 14336: T = 320, 384 11% faster,
    // T = 512 and 1024 8%).
    const int64_t large_tiles = cdiv(T, GateUpLarge::BN) * cdiv(F, GateUpLarge::BMW);
    if (large_tiles >= 512 || (T > 256 && large_tiles >= 192))
        gemm_step<GateUpLarge>(p.gate_up, K_GEMM_GU_L, (int)F, (int)T, (int)D, 2, false, kGroupGateUp);
    else if (T <= GateUpTiny::BN)
        gemm_step<GateUpTiny>(p.gate_up, K_GEMM_GU_T, (int)F, (int)T, (int)D, 2, true, kGroupGateUp);
    else if (T <= GateUpMid::BN)
        gemm_step<GateUpMid>(p.gate_up, K_GEMM_GU_M, (int)F, (int)T, (int)D, 2, true, kGroupGateUp);
    else
        gemm_step<GateUpSmall>(p.gate_up, K_GEMM_GU_S, (int)F, (int)T, (int)D, 2, true, kGroupGateUp);
    if (cdiv(T, DownLarge::BN) * cdiv(D, DownLarge::BMW) >= 192)
        gemm_step<DownLarge>(p.down, K_GEMM_DN_L, (int)D, (int)T, (int)F, 1, false, kGroupDown);
    else if (T <= DownTiny::BN)
        gemm_step<DownTiny>(p.down, K_GEMM_DN_T, (int)D, (int)T, (int)F, 1, true, kGroupDown);
    else if (T <= DownMid::BN)
        gemm_step<DownMid>(p.down, K_GEMM_DN_M, (int)D, (int)T, (int)F, 1, true, kGroupDown);
    else
        gemm_step<DownSmall>(p.down, K_GEMM_DN_S, (int)D, (int)T, (int)F, 1, true, kGroupDown);
    return p;
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
        counters = std::max({counters, p.gate_up.counters, p.down.counters});
        partial = std::max({partial, p.gate_up.partial_bytes, p.down.partial_bytes});
        if (path == GMLP_PATH_GEMV) // the fused kernel runs both steps at once: separate partial sums
            partial = std::max(partial, align_up(p.gate_up.partial_bytes) + p.down.partial_bytes);
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
    if (D > kMaxDim || F > kMaxDim || T > kMaxTokens)
        return fail(GMLP_ERR_UNSUPPORTED, "shape T=%lld D=%lld F=%lld exceeds the supported range "
                    "(D, F <= %lld, T <= %lld)", (long long)T, (long long)D, (long long)F,
                    (long long)kMaxDim, (long long)kMaxTokens);
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

int hip_check(hipError_t e, const char *what)
{
    if (e != hipSuccess)
        return fail(GMLP_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return GMLP_OK;
}

// ---- launches ----------------------------------------------------------------

// Weights are streamed (nontemporal loads) when the plan has a single token
// tile: then each weight element is read by one block only.
bool stream_weights(const Step &s) { return s.tiles_n == 1; }

template <class S, int EPI, bool SPLIT, bool STREAM_W = false>
int launch_gemm(const Step &s, const void *w0, const void *w1, const void *act, void *out,
                uint8_t *ws, const Layout &l, const Variant &v, const float *rrms, const float *rowdiv,
                hipStream_t stream)
{
    GemmParams p;
    p.w0 = static_cast<const uint16_t *>(w0);
    p.w1 = static_cast<const uint16_t *>(w1);
    p.act = static_cast<const uint16_t *>(act);
    p.out = static_cast<uint16_t *>(out);
    p.partial = reinterpret_cast<float *>(ws + l.partial_off);
    p.counters = reinterpret_cast<uint32_t *>(ws + l.counters_off);
    p.M = s.M;
    p.N = s.N;
    p.K = s.K;
    p.k_split = s.k_split;
    p.splits = s.splits;
    p.tiles_m = s.tiles_m;
    p.tiles_n = s.tiles_n;
    p.group_m = s.group_m;
    p.tile_base = s.tile_base;
    p.tile_count = s.tile_count;
    p.activation = v.act;
    p.beta = v.beta;
    p.rrms = rrms;
    p.rowdiv = rowdiv;
    if (!SPLIT && s.splits != 1)
        return fail(GMLP_ERR_INVALID_ARG, "internal: split-K plan for a kernel without split-K");
    if (s.partial_bytes > (size_t)kNumRecords)
        return fail(GMLP_ERR_UNSUPPORTED, "split-K partial sums of %zu bytes exceed the 2 GiB buffer range",
                    s.partial_bytes);
    hipLaunchKernelGGL((gemm_mfma_kernel<S, EPI, SPLIT, STREAM_W>), dim3(s.blocks), dim3(S::NTHREADS), 0, stream, p);
    return hip_check(hipGetLastError(), "MFMA GEMM launch");
}

GemvParams gemv_params(const Step &s, const void *w0, const void *w1, const void *act, void *out,
                       uint8_t *ws, const Layout &l, const Variant &v, const float *rowdiv)
{
    GemvParams p;
    p.w0 = static_cast<const uint16_t *>(w0);
    p.w1 = static_cast<const uint16_t *>(w1);
    p.act = static_cast<const uint16_t *>(act);
    p.out = static_cast<uint16_t *>(out);
    p.partial = reinterpret_cast<float *>(ws + l.partial_off);
    p.counters = reinterpret_cast<uint32_t *>(ws + l.counters_off);
    p.M = s.M;
    p.K = s.K;
    p.k_split = s.k_split;
    p.splits = s.splits;
    p.strips = s.strips;
    p.strip_lanes = s.strip_lanes;
    p.activation = v.act;
    p.beta = v.beta;
    p.eps = v.eps;
    // Sums of squares follow the column sums of every split.
    p.ssq = p.partial + (size_t)s.splits * 2 * s.N * s.M;
    p.rowdiv = rowdiv;
    return p;
}

template <int NT, int NW, int EPI, bool RMS>
int launch_gemv_nt(const Step &s, const void *w0, const void *w1, const void *act, void *out,
                   uint8_t *ws, const Layout &l, const Variant &v, const float *rowdiv, hipStream_t stream)
{
    const GemvParams p = gemv_params(s, w0, w1, act, out, ws, l, v, rowdiv);
    hipLaunchKernelGGL((gemv_splitk_kernel<NT, NW, EPI, RMS>), dim3(s.blocks), dim3(kGemvThreads), 0,
                       stream, p);
    return hip_check(hipGetLastError(), "GEMV launch");
}

template <int NW, int EPI, bool RMS>
int launch_gemv(const Step &s, const void *w0, const void *w1, const void *act, void *out,
                uint8_t *ws, const Layout &l, const Variant &v, hipStream_t stream,
                const float *rowdiv = nullptr)
{
    switch (s.N) {
    case 1: return launch_gemv_nt<1, NW, EPI, RMS>(s, w0, w1, act, out, ws, l, v, rowdiv, stream);
    case 2: return launch_gemv_nt<2, NW, EPI, RMS>(s, w0, w1, act, out, ws, l, v, rowdiv, stream);
    case 3: return launch_gemv_nt<3, NW, EPI, RMS>(s, w0, w1, act, out, ws, l, v, rowdiv, stream);
    case 4: return launch_gemv_nt<4, NW, EPI, RMS>(s, w0, w1, act, out, ws, l, v, rowdiv, stream);
    case 5: return launch_gemv_nt<5, NW, EPI, RMS>(s, w0, w1, act, out, ws, l, v, rowdiv, stream);
    case 6: return launch_gemv_nt<6, NW, EPI, RMS>(s, w0, w1, act, out, ws, l, v, rowdiv, stream);
    case 7: return launch_gemv_nt<7, NW, EPI, RMS>(s, w0, w1, act, out, ws, l, v, rowdiv, stream);
    case 8: return launch_gemv_nt<8, NW, EPI, RMS>(s, w0, w1, act, out, ws, l, v, rowdiv, stream);
    default: return fail(GMLP_ERR_INVALID_ARG, "GEMV path needs 1 <= T <= 8 (T=%d)", s.N);
    }
}

// The gate/up step: H = bf16(act(r G) * (r U)).  With RMSNorm the GEMV
// kernel computes r itself; the MFMA path computes r for every row first.
int run_gate_up(const Step &s, const void *X, const void *Wg, const void *Wu, void *H, uint8_t *ws,
                const Layout &l, const Variant &v, hipStream_t st)
{
    const float *rrms = nullptr;
    if (v.rms && s.kind != K_GEMV) {
        float *r = reinterpret_cast<float *>(ws + l.rrms_off);
        const int per = kRowRmsThreads / 64;
        hipLaunchKernelGGL(row_rms_kernel, dim3((unsigned)cdiv(s.N, per)), dim3(kRowRmsThreads), 0, st,
                           static_cast<const uint16_t *>(X), r, s.N, s.K, v.eps);
        int rc = hip_check(hipGetLastError(), "row RMS launch");
        if (rc)
            return rc;
        rrms = r;
    }
    switch (s.kind) {
    case K_GEMM_GU_L: {
        const int rc = launch_gemm<GateUpLarge, EPI_GATE_MUL, false>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
        if (rc || !s.tail_tiles)
            return rc;
        return launch_gemm<GateUpLarge, EPI_GATE_MUL, true>(tail_step(s), Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
    }
    case K_GEMM_GU_S:
        return stream_weights(s) ? launch_gemm<GateUpSmall, EPI_GATE_MUL, true, true>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st)
                                 : launch_gemm<GateUpSmall, EPI_GATE_MUL, true, false>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
    case K_GEMM_GU_T: // one token tile: always streamed
        return launch_gemm<GateUpTiny, EPI_GATE_MUL, true, true>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
    case K_GEMM_GU_M:
        return stream_weights(s) ? launch_gemm<GateUpMid, EPI_GATE_MUL, true, true>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st)
                                 : launch_gemm<GateUpMid, EPI_GATE_MUL, true, false>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
    case K_GEMV:
        return v.rms ? launch_gemv<2, EPI_GATE_MUL, true>(s, Wg, Wu, X, H, ws, l, v, st)
                     : launch_gemv<2, EPI_GATE_MUL, false>(s, Wg, Wu, X, H, ws, l, v, st);
    default: return fail(GMLP_ERR_INVALID_ARG, "no gate/up kernel for this plan");
    }
}

// The down step, Y = bf16(H Wd), or with row divisors d, Y = bf16((H Wd) / d)
// row by row (the divide of Softmax+MatMul moved past its matmul).
int run_down(const Step &s, const void *H, const void *Wd, void *Y, uint8_t *ws, const Layout &l,
             hipStream_t st, const float *rowdiv = nullptr)
{
    const Variant plain;
    switch (s.kind) {
    case K_GEMM_DN_L: {
        const int rc = launch_gemm<DownLarge, EPI_STORE, false>(s, Wd, nullptr, H, Y, ws, l, plain, nullptr, rowdiv,
                                                                 st);
        if (rc || !s.tail_tiles)
            return rc;
        return launch_gemm<DownLarge, EPI_STORE, true>(tail_step(s), Wd, nullptr, H, Y, ws, l, plain, nullptr,
                                                        rowdiv, st);
    }
    case K_GEMM_DN_S:
        return stream_weights(s) ? launch_gemm<DownSmall, EPI_STORE, true, true>(s, Wd, nullptr, H, Y, ws, l, plain,
                                                                                 nullptr, rowdiv, st)
                                 : launch_gemm<DownSmall, EPI_STORE, true, false>(s, Wd, nullptr, H, Y, ws, l, plain,
                                                                                  nullptr, rowdiv, st);
    case K_GEMM_DN_T: // one token tile: always streamed
        return launch_gemm<DownTiny, EPI_STORE, true, true>(s, Wd, nullptr, H, Y, ws, l, plain, nullptr, rowdiv, st);
    case K_GEMM_DN_M:
        return stream_weights(s) ? launch_gemm<DownMid, EPI_STORE, true, true>(s, Wd, nullptr, H, Y, ws, l, plain,
                                                                               nullptr, rowdiv, st)
                                 : launch_gemm<DownMid, EPI_STORE, true, false>(s, Wd, nullptr, H, Y, ws, l, plain,
                                                                                nullptr, rowdiv, st);
    case K_GEMV: return launch_gemv<1, EPI_STORE, false>(s, Wd, nullptr, H, Y, ws, l, plain, st, rowdiv);
    default: return fail(GMLP_ERR_INVALID_ARG, "no down kernel for this plan");
    }
}

// The fused kernel: the gate/up items on the first blocks, the down items on
// the rest, all in one launch.
int fused_grid(const Plan &plan) { return plan.gate_up.blocks + plan.down.blocks; }

template <int NT, bool RMS>
int launch_fused_nt(const Plan &plan, const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y,
                    uint8_t *ws, const Layout &l, const Variant &v, hipStream_t st)
{
    if (plan.down.splits > kFusedMaxSplits)
        return fail(GMLP_ERR_UNSUPPORTED, "fused path: %d down splits, at most %d", plan.down.splits,
                    kFusedMaxSplits);
    if ((size_t)(plan.gate_up.strips + plan.down.strips) * sizeof(uint32_t) > kStripCounterBytes)
        return fail(GMLP_ERR_UNSUPPORTED, "fused path: too many strips for the counter block");
    void *H = ws + l.h_off;
    GemvFusedParams fp;
    fp.gate_up = gemv_params(plan.gate_up, Wg, Wu, X, H, ws, l, v, nullptr);
    fp.down = gemv_params(plan.down, Wd, nullptr, H, Y, ws, l, Variant{}, nullptr);
    fp.down.counters = fp.gate_up.counters + plan.gate_up.strips;
    fp.down.partial = reinterpret_cast<float *>(ws + l.partial_off + align_up(plan.gate_up.partial_bytes));
    fp.ready = reinterpret_cast<uint32_t *>(ws + l.counters_off + kStripCounterBytes);
    fp.errors = reinterpret_cast<uint32_t *>(ws + l.counters_off + kErrorOffset);
    fp.spin_limit = g_spin_limit.load();
    hipLaunchKernelGGL((gemv_fused_kernel<NT, RMS>), dim3(fused_grid(plan)), dim3(kGemvThreads), 0, st, fp);
    return hip_check(hipGetLastError(), "fused kernel launch");
}

template <bool RMS>
int launch_fused(const Plan &plan, const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y,
                 uint8_t *ws, const Layout &l, const Variant &v, hipStream_t st)
{
    switch (plan.gate_up.N) {
    case 1: return launch_fused_nt<1, RMS>(plan, X, Wg, Wu, Wd, Y, ws, l, v, st);
    case 2: return launch_fused_nt<2, RMS>(plan, X, Wg, Wu, Wd, Y, ws, l, v, st);
    case 3: return launch_fused_nt<3, RMS>(plan, X, Wg, Wu, Wd, Y, ws, l, v, st);
    case 4: return launch_fused_nt<4, RMS>(plan, X, Wg, Wu, Wd, Y, ws, l, v, st);
    case 5: return launch_fused_nt<5, RMS>(plan, X, Wg, Wu, Wd, Y, ws, l, v, st);
    case 6: return launch_fused_nt<6, RMS>(plan, X, Wg, Wu, Wd, Y, ws, l, v, st);
    case 7: return launch_fused_nt<7, RMS>(plan, X, Wg, Wu, Wd, Y, ws, l, v, st);
    case 8: return launch_fused_nt<8, RMS>(plan, X, Wg, Wu, Wd, Y, ws, l, v, st);
    default: return fail(GMLP_ERR_INVALID_ARG, "fused path needs 1 <= T <= 8 (T=%d)", plan.gate_up.N);
    }
}

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
    if (path != GMLP_PATH_AUTO && path != GMLP_PATH_GEMV && path != GMLP_PATH_MFMA && path != GMLP_PATH_FUSED)
        return fail(GMLP_ERR_INVALID_ARG, "unknown path %d", path);
    if ((path == GMLP_PATH_GEMV || path == GMLP_PATH_FUSED) && T > kGemvMaxTokens)
        return fail(GMLP_ERR_UNSUPPORTED, "%s path needs T <= %d (T=%lld)",
                    path == GMLP_PATH_GEMV ? "GEMV" : "fused", kGemvMaxTokens, (long long)T);
    return GMLP_OK;
}

// The entry points that run one step alone (and Softmax+MatMul) have no
// fused form.
int check_single_step_path(int path, int64_t T)
{
    if (path == GMLP_PATH_FUSED)
        return fail(GMLP_ERR_UNSUPPORTED, "the fused path runs the whole Gated MLP only");
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

// Stream-ordered scratch for the entry points that allocate.
struct Scratch {
    void *ptr = nullptr;
    hipStream_t stream = nullptr;
    ~Scratch()
    {
        if (ptr)
            (void)hipFreeAsync(ptr, stream);
    }
    int alloc(size_t bytes, const Layout &l, hipStream_t st)
    {
        stream = st;
        int rc = hip_check(hipMallocAsync(&ptr, bytes, st), "hipMallocAsync(workspace)");
        if (rc) {
            ptr = nullptr;
            return rc == GMLP_ERR_HIP ? fail(GMLP_ERR_NO_MEMORY, "%s", g_err) : rc;
        }
        return hip_check(hipMemsetAsync(ptr, 0, l.h_off, st), "hipMemsetAsync(counters)");
    }
};

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
    case K_GEMM_DN_L: return "gemm_mfma_kernel<" + shape_name<DownLarge>() + ", 1, false, false>";
    case K_GEMM_DN_S:
        return "gemm_mfma_kernel<" + shape_name<DownSmall>() + ", 1, true, " + (stream_weights(s) ? "true>" : "false>");
    case K_GEMM_GU_T: return "gemm_mfma_kernel<" + shape_name<GateUpTiny>() + ", 0, true, true>";
    case K_GEMM_DN_T: return "gemm_mfma_kernel<" + shape_name<DownTiny>() + ", 1, true, true>";
    case K_GEMM_GU_M:
        return "gemm_mfma_kernel<" + shape_name<GateUpMid>() + ", 0, true, " + (stream_weights(s) ? "true>" : "false>");
    case K_GEMM_DN_M:
        return "gemm_mfma_kernel<" + shape_name<DownMid>() + ", 1, true, " + (stream_weights(s) ? "true>" : "false>");
    case K_GEMV:
        return "gemv_splitk_kernel<" + std::to_string(s.N) + (gate_up ? ", 2, 0, false>" : ", 1, 1, false>");
    default: return "none";
    }
}

// The describe lines of a step: its launch, then its tail launch if any.
std::string describe_step(const Step &s, bool gate_up)
{
    char tmp[200];
    snprintf(tmp, sizeof tmp, "%s grid=%d block=%d k_splits=%d\n", kernel_name(s, gate_up).c_str(), s.blocks,
             s.threads, s.splits);
    std::string text = tmp;
    if (s.tail_tiles) {
        const Step t = tail_step(s);
        const std::string shape = s.kind == K_GEMM_GU_L ? shape_name<GateUpLarge>() + ", 0" : shape_name<DownLarge>() + ", 1";
        snprintf(tmp, sizeof tmp, "gemm_mfma_kernel<%s, true, false> grid=%d block=%d k_splits=%d\n", shape.c_str(),
                 t.blocks, t.threads, t.splits);
        text += tmp;
    }
    return text;
}

} // namespace

extern "C" {

int gmlp_version(void) { return GMLP_VERSION; }

const char *gmlp_status_string(int status)
{
    switch (status) {
    case GMLP_OK: return "GMLP_OK";
    case GMLP_ERR_INVALID_ARG: return "GMLP_ERR_INVALID_ARG";
    case GMLP_ERR_UNSUPPORTED: return "GMLP_ERR_UNSUPPORTED";
    case GMLP_ERR_HIP: return "GMLP_ERR_HIP";
    case GMLP_ERR_NO_MEMORY: return "GMLP_ERR_NO_MEMORY";
    default: return "GMLP_ERR_UNKNOWN";
    }
}

const char *gmlp_last_error(void) { return g_err; }

int gmlp_validate(int64_t T, int64_t D, int64_t F, const void *X, const void *Wg, const void *Wu,
                  const void *Wd, const void *Y)
{
    int rc = validate(T, D, F, X, Wg, Wu, Wd, Y);
    return rc ? rc : ok();
}

int gmlp_describe(int64_t T, int64_t D, int64_t F, int path, char *buf, size_t bytes)
{
    int rc;
    if (!buf || !bytes)
        return fail(GMLP_ERR_INVALID_ARG, "describe needs a buffer");
    buf[0] = '\0';
    if ((rc = check_shape(T, D, F)) || (rc = check_path(path, T)))
        return rc;
    if (T == 0)
        return ok();
    const Plan plan = make_plan(T, D, F, path);
    std::string text;
    auto line = [&](const char *name, int blocks, int threads, int splits) {
        char tmp[160];
        snprintf(tmp, sizeof tmp, "%s grid=%d block=%d k_splits=%d\n", name, blocks, threads, splits);
        text += tmp;
    };
    if (plan.path == GMLP_PATH_FUSED) {
        const std::string name = "gemv_fused_kernel<" + std::to_string(T) + ", false>";
        line(name.c_str(), fused_grid(plan), kGemvThreads, plan.gate_up.splits);
        snprintf(buf, bytes, "%s", text.c_str());
        return ok();
    }
    for (const Step *s : {&plan.gate_up, &plan.down})
        text += describe_step(*s, s == &plan.gate_up);
    snprintf(buf, bytes, "%s", text.c_str());
    return ok();
}

size_t gmlp_workspace_size(int64_t T, int64_t D, int64_t F)
{
    if (check_shape(T, D, F))
        return 0;
    return make_layout(T, D, F).total;
}

int gmlp_workspace_init(void *workspace, size_t bytes, void *stream)
{
    if (!workspace)
        return fail(GMLP_ERR_INVALID_ARG, "workspace is NULL");
    // Only the counter block at the start must be zero.
    const size_t n = std::min(bytes, kCounterBytes);
    int rc = hip_check(hipMemsetAsync(workspace, 0, n, static_cast<hipStream_t>(stream)),
                       "hipMemsetAsync(workspace)");
    return rc ? rc : ok();
}

int gmlp_workspace_status(void *workspace, size_t bytes, void *stream, uint32_t *fused_giveups)
{
    int rc;
    if (!workspace || !fused_giveups)
        return fail(GMLP_ERR_INVALID_ARG, "workspace and fused_giveups must not be NULL");
    if (bytes < kCounterBytes)
        return fail(GMLP_ERR_INVALID_ARG, "a workspace of %zu bytes has no status word (%zu needed)", bytes,
                    kCounterBytes);
    hipStream_t st = static_cast<hipStream_t>(stream);
    uint32_t *word = reinterpret_cast<uint32_t *>(static_cast<uint8_t *>(workspace) + kErrorOffset);
    uint32_t host = 0;
    if ((rc = hip_check(hipMemcpyAsync(&host, word, sizeof host, hipMemcpyDeviceToHost, st),
                        "hipMemcpyAsync(status)")) ||
        (rc = hip_check(hipStreamSynchronize(st), "hipStreamSynchronize")))
        return rc;
    if (host && ((rc = hip_check(hipMemsetAsync(word, 0, sizeof host, st), "hipMemsetAsync(status)")) ||
                 (rc = hip_check(hipStreamSynchronize(st), "hipStreamSynchronize"))))
        return rc;
    *fused_giveups = host;
    return ok();
}

uint32_t gmlp_test_fused_spin_limit(uint32_t limit) { return g_spin_limit.exchange(limit); }

int gmlp_forward_variant(const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y, int64_t T,
                         int64_t D, int64_t F, int activation, float beta, int rmsnorm, float eps,
                         int path, void *workspace, size_t ws_bytes, void *stream)
{
    int rc;
    Variant v;
    if ((rc = validate(T, D, F, X, Wg, Wu, Wd, Y)) || (rc = check_path(path, T)) ||
        (rc = check_variant(activation, beta, rmsnorm, eps, &v)))
        return rc;
    if (T == 0)
        return ok();
    const Layout l = make_layout(T, D, F);
    if ((rc = check_workspace(workspace, ws_bytes, l)))
        return rc;
    const Plan plan = make_plan(T, D, F, path);
    uint8_t *ws = static_cast<uint8_t *>(workspace);
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (plan.path == GMLP_PATH_FUSED) {
        rc = v.rms ? launch_fused<true>(plan, X, Wg, Wu, Wd, Y, ws, l, v, st)
                   : launch_fused<false>(plan, X, Wg, Wu, Wd, Y, ws, l, v, st);
        return rc ? rc : ok();
    }
    void *H = ws + l.h_off;
    if ((rc = run_gate_up(plan.gate_up, X, Wg, Wu, H, ws, l, v, st)) ||
        (rc = run_down(plan.down, H, Wd, Y, ws, l, st)))
        return rc;
    return ok();
}

int gmlp_forward_ex(const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y, int64_t T,
                    int64_t D, int64_t F, int path, void *workspace, size_t ws_bytes, void *stream)
{
    return gmlp_forward_variant(X, Wg, Wu, Wd, Y, T, D, F, GMLP_ACT_SILU, 1.0f, 0, 0.0f, path, workspace,
                                ws_bytes, stream);
}

int gmlp_forward_ws(const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y, int64_t T,
                    int64_t D, int64_t F, void *workspace, size_t ws_bytes, void *stream)
{
    return gmlp_forward_ex(X, Wg, Wu, Wd, Y, T, D, F, GMLP_PATH_AUTO, workspace, ws_bytes, stream);
}

int gmlp_forward(const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y, int64_t T,
                 int64_t D, int64_t F, void *stream)
{
    int rc;
    if ((rc = validate(T, D, F, X, Wg, Wu, Wd, Y)))
        return rc;
    if (T == 0)
        return ok();
    const Layout l = make_layout(T, D, F);
    Scratch s;
    if ((rc = s.alloc(l.total, l, static_cast<hipStream_t>(stream))))
        return rc;
    return gmlp_forward_ex(X, Wg, Wu, Wd, Y, T, D, F, GMLP_PATH_AUTO, s.ptr, l.total, stream);
}

} // extern "C"

// ---- the entry point that allocates nothing -------------------------------------
// gmlp_forward_noalloc keeps its workspace (counter block, H, split-K partial
// sums) in this array.  Every device the library runs on holds its own copy
// from the moment the library's code is loaded on it until the process ends.
// In host code `scratch` names a host-side stand-in, not device memory: only
// the per-device address from hipGetSymbolAddress may be handed to kernels.
static __device__ __align__(256) uint8_t scratch[GMLP_NOALLOC_SCRATCH_BYTES];

namespace {

// Zero n 32-bit words (the counter block of the scratch array at set-up).
__global__ void zero_words_kernel(uint32_t *p, uint32_t n)
{
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        p[i] = 0u;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t *g_scratch_ptr[kMaxDevices]; // device address of `scratch` per device (nullptr: not set up)

// The current device's copy of `scratch`.  Set-up, once per device with that
// device current: take the array's device address and zero its counter block
// with a kernel on `st` (ordered before the caller's kernels on that stream;
// the kernels leave the counters at zero when they finish, so later calls
// find them zero).
int noalloc_scratch(hipStream_t st, uint8_t **out)
{
    int dev = -1, rc;
    if ((rc = hip_check(hipGetDevice(&dev), "hipGetDevice")))
        return rc;
    if (dev < 0 || dev >= kMaxDevices)
        return fail(GMLP_ERR_UNSUPPORTED, "device %d: gmlp_forward_noalloc supports devices 0..%d", dev,
                    kMaxDevices - 1);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        if ((rc = hip_check(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)")))
            return rc;
        const uint32_t words = (uint32_t)(kCounterBytes / sizeof(uint32_t));
        hipLaunchKernelGGL(zero_words_kernel, dim3(64), dim3(256), 0, st, static_cast<uint32_t *>(p), words);
        if ((rc = hip_check(hipGetLastError(), "scratch counter clear launch")))
            return rc;
        g_scratch_ptr[dev] = static_cast<uint8_t *>(p);
    }
    *out = g_scratch_ptr[dev];
    return GMLP_OK;
}

} // namespace

extern "C" int gmlp_forward_noalloc(const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y,
                                    int64_t T, int64_t D, int64_t F, void *stream)
{
    int rc;
    if ((rc = validate(T, D, F, X, Wg, Wu, Wd, Y)))
        return rc;
    if (T == 0)
        return ok();
    const Layout l = make_layout(T, D, F);
    if (l.total > (size_t)GMLP_NOALLOC_SCRATCH_BYTES)
        return fail(GMLP_ERR_UNSUPPORTED,
                    "shape T=%lld D=%lld F=%lld needs %zu bytes of scratch, more than the %zu bytes "
                    "gmlp_forward_noalloc holds (use gmlp_forward_ws with a caller workspace)",
                    (long long)T, (long long)D, (long long)F, l.total, (size_t)GMLP_NOALLOC_SCRATCH_BYTES);
    const hipStream_t st = static_cast<hipStream_t>(stream);
    uint8_t *ws = nullptr;
    if ((rc = noalloc_scratch(st, &ws)))
        return rc;
    return gmlp_forward_ex(X, Wg, Wu, Wd, Y, T, D, F, GMLP_PATH_AUTO, ws, (size_t)GMLP_NOALLOC_SCRATCH_BYTES,
                           stream);
}

namespace {

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

} // namespace

extern "C" {

int gmlp_gate_up_variant(const void *X, const void *Wg, const void *Wu, void *H, int64_t T, int64_t D,
                         int64_t F, int activation, float beta, int rmsnorm, float eps, int path,
                         void *workspace, size_t ws_bytes, void *stream)
{
    int rc;
    Variant v;
    if ((rc = check_gate_up_args(X, Wg, Wu, H, T, D, F)) || (rc = check_single_step_path(path, T)) ||
        (rc = check_variant(activation, beta, rmsnorm, eps, &v)))
        return rc;
    if (T == 0)
        return ok();
    const Layout l = make_layout(T, D, F);
    if ((rc = check_workspace(workspace, ws_bytes, l)))
        return rc;
    const Plan plan = make_plan(T, D, F, path);
    if ((rc = run_gate_up(plan.gate_up, X, Wg, Wu, H, static_cast<uint8_t *>(workspace), l, v,
                          static_cast<hipStream_t>(stream))))
        return rc;
    return ok();
}

int gmlp_gate_up_ws(const void *X, const void *Wg, const void *Wu, void *H, int64_t T, int64_t D,
                    int64_t F, int path, void *workspace, size_t ws_bytes, void *stream)
{
    return gmlp_gate_up_variant(X, Wg, Wu, H, T, D, F, GMLP_ACT_SILU, 1.0f, 0, 0.0f, path, workspace,
                                ws_bytes, stream);
}

int gmlp_down_ws(const void *H, const void *Wd, void *Y, int64_t T, int64_t F, int64_t D, int path,
                 void *workspace, size_t ws_bytes, void *stream)
{
    int rc;
    if ((rc = check_down_args(H, Wd, Y, T, F, D)) || (rc = check_single_step_path(path, T)))
        return rc;
    if (T == 0)
        return ok();
    const Layout l = make_layout(T, D, F);
    if ((rc = check_workspace(workspace, ws_bytes, l)))
        return rc;
    const Plan plan = make_plan(T, D, F, path);
    if ((rc = run_down(plan.down, H, Wd, Y, static_cast<uint8_t *>(workspace), l,
                       static_cast<hipStream_t>(stream))))
        return rc;
    return ok();
}

int gmlp_gate_up(const void *X, const void *Wg, const void *Wu, void *H, int64_t T, int64_t D,
                 int64_t F, void *stream)
{
    int rc;
    if ((rc = check_gate_up_args(X, Wg, Wu, H, T, D, F)))
        return rc;
    if (T == 0)
        return ok();
    const Layout l = make_layout(T, D, F);
    Scratch s;
    if ((rc = s.alloc(l.total, l, static_cast<hipStream_t>(stream))))
        return rc;
    return gmlp_gate_up_ws(X, Wg, Wu, H, T, D, F, GMLP_PATH_AUTO, s.ptr, l.total, stream);
}

int gmlp_down(const void *H, const void *Wd, void *Y, int64_t T, int64_t F, int64_t D, void *stream)
{
    int rc;
    if ((rc = check_down_args(H, Wd, Y, T, F, D)))
        return rc;
    if (T == 0)
        return ok();
    const Layout l = make_layout(T, D, F);
    Scratch s;
    if ((rc = s.alloc(l.total, l, static_cast<hipStream_t>(stream))))
        return rc;
    return gmlp_down_ws(H, Wd, Y, T, F, D, GMLP_PATH_AUTO, s.ptr, l.total, stream);
}

} // extern "C"

// ---- Softmax+MatMul --------------------------------------------------------------
// Z = softmax(X) Y computed as (P Y) / s: softmax_exp_rows_kernel writes
// P = exp(X - rowmax) and the row sums s, then the Gated MLP's down-step
// kernels (T = M tokens, F = K contracted rows, D = N output columns) run the
// matmul with s as the row divisors of their epilogue.

namespace {

int check_smm_shape(int64_t M, int64_t K, int64_t N)
{
    if (M < 0 || K <= 0 || N <= 0)
        return fail(GMLP_ERR_INVALID_ARG, "invalid shape M=%lld K=%lld N=%lld (need M >= 0, K > 0, N > 0)",
                    (long long)M, (long long)K, (long long)N);
    if (K % 8 || N % 8)
        return fail(GMLP_ERR_UNSUPPORTED, "K=%lld and N=%lld must be multiples of 8", (long long)K,
                    (long long)N);
    if (K > kMaxDim || N > kMaxDim || M > kMaxTokens)
        return fail(GMLP_ERR_UNSUPPORTED, "shape M=%lld K=%lld N=%lld exceeds the supported range "
                    "(K, N <= %lld, M <= %lld)", (long long)M, (long long)K, (long long)N,
                    (long long)kMaxDim, (long long)kMaxTokens);
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

int launch_softmax_rows(const void *X, uint16_t *P, float *sums, int64_t M, int64_t K, hipStream_t st)
{
    const dim3 grid((unsigned)cdiv(M, kSoftmaxThreads / 64)), block(kSoftmaxThreads);
    const uint16_t *x = static_cast<const uint16_t *>(X);
    switch (softmax_chunks_per_lane((int)K)) {
    case 1: hipLaunchKernelGGL(softmax_exp_rows_kernel<1>, grid, block, 0, st, x, P, sums, (int)M, (int)K); break;
    case 2: hipLaunchKernelGGL(softmax_exp_rows_kernel<2>, grid, block, 0, st, x, P, sums, (int)M, (int)K); break;
    case 4: hipLaunchKernelGGL(softmax_exp_rows_kernel<4>, grid, block, 0, st, x, P, sums, (int)M, (int)K); break;
    case 8: hipLaunchKernelGGL(softmax_exp_rows_kernel<8>, grid, block, 0, st, x, P, sums, (int)M, (int)K); break;
    default:
        hipLaunchKernelGGL(softmax_exp_rows_kernel<kSoftmaxMaxChunks>, grid, block, 0, st, x, P, sums, (int)M,
                           (int)K);
        break;
    }
    return hip_check(hipGetLastError(), "softmax exp/row-sum launch");
}

} // namespace

extern "C" {

size_t softmax_matmul_workspace_size(int64_t M, int64_t K, int64_t N)
{
    if (check_smm_shape(M, K, N))
        return 0;
    return smm_layout(M, K, N).total;
}

int softmax_matmul_describe(int64_t M, int64_t K, int64_t N, int path, char *buf, size_t bytes)
{
    int rc;
    if (!buf || !bytes)
        return fail(GMLP_ERR_INVALID_ARG, "describe needs a buffer");
    buf[0] = '\0';
    if ((rc = check_smm_shape(M, K, N)))
        return rc;
    if ((rc = check_single_step_path(path, M)))
        return rc;
    if (M == 0)
        return ok();
    const Step s = smm_matmul_step(M, K, N, path);
    const int r = softmax_chunks_per_lane((int)K);
    snprintf(buf, bytes, "softmax_exp_rows_kernel<%d> grid=%lld block=%d k_splits=1\n%s", r,
             (long long)cdiv(M, kSoftmaxThreads / 64), kSoftmaxThreads, describe_step(s, false).c_str());
    return ok();
}

int softmax_matmul_ws(const void *X, const void *Y, void *Z, int64_t M, int64_t K, int64_t N, int path,
                      void *workspace, size_t ws_bytes, void *stream)
{
    int rc;
    if ((rc = check_smm_args(X, Y, Z, M, K, N)) || (rc = check_single_step_path(path, M)))
        return rc;
    if (M == 0)
        return ok();
    const Layout l = smm_layout(M, K, N);
    if ((rc = check_workspace(workspace, ws_bytes, l)))
        return rc;
    if (overlaps(Z, (size_t)M * N * 2, workspace, l.total))
        return fail(GMLP_ERR_INVALID_ARG, "Z overlaps the workspace");
    uint8_t *ws = static_cast<uint8_t *>(workspace);
    hipStream_t st = static_cast<hipStream_t>(stream);
    uint16_t *P = reinterpret_cast<uint16_t *>(ws + l.h_off);
    float *sums = reinterpret_cast<float *>(ws + l.rrms_off);
    const Step s = smm_matmul_step(M, K, N, path);
    if ((rc = launch_softmax_rows(X, P, sums, M, K, st)) || (rc = run_down(s, P, Y, Z, ws, l, st, sums)))
        return rc;
    return ok();
}

int softmax_matmul_exp_rows(const void *X, void *P, float *s, int64_t M, int64_t K, void *stream)
{
    int rc;
    if ((rc = check_smm_shape(M, K, 8)) || (rc = check_ptr(X, "X", M > 0)) || (rc = check_ptr(P, "P", M > 0)))
        return rc;
    if (M > 0 && !s)
        return fail(GMLP_ERR_INVALID_ARG, "s is NULL");
    if (reinterpret_cast<uintptr_t>(s) % 4)
        return fail(GMLP_ERR_UNSUPPORTED, "s (%p) is not 4-byte aligned", (const void *)s);
    const size_t xb = (size_t)M * K * 2, sb = (size_t)M * sizeof(float);
    if (overlaps(P, xb, X, xb) || overlaps(s, sb, X, xb) || overlaps(s, sb, P, xb))
        return fail(GMLP_ERR_INVALID_ARG, "X, P and s must not overlap");
    if (M == 0)
        return ok();
    if ((rc = launch_softmax_rows(X, static_cast<uint16_t *>(P), s, M, K, static_cast<hipStream_t>(stream))))
        return rc;
    return ok();
}

int softmax_matmul_divide_ws(const void *P, const float *s, const void *Y, void *Z, int64_t M, int64_t K,
                             int64_t N, int path, void *workspace, size_t ws_bytes, void *stream)
{
    int rc;
    if ((rc = check_smm_args(P, Y, Z, M, K, N)) || (rc = check_single_step_path(path, M)))
        return rc;
    if (M > 0 && !s)
        return fail(GMLP_ERR_INVALID_ARG, "s is NULL");
    if (reinterpret_cast<uintptr_t>(s) % 4)
        return fail(GMLP_ERR_UNSUPPORTED, "s (%p) is not 4-byte aligned", (const void *)s);
    if (overlaps(Z, (size_t)M * N * 2, s, (size_t)M * sizeof(float)))
        return fail(GMLP_ERR_INVALID_ARG, "Z overlaps s");
    if (M == 0)
        return ok();
    const Layout l = smm_layout(M, K, N);
    if ((rc = check_workspace(workspace, ws_bytes, l)))
        return rc;
    if (overlaps(Z, (size_t)M * N * 2, workspace, l.total))
        return fail(GMLP_ERR_INVALID_ARG, "Z overlaps the workspace");
    const Step st = smm_matmul_step(M, K, N, path);
    if ((rc = run_down(st, P, Y, Z, static_cast<uint8_t *>(workspace), l, static_cast<hipStream_t>(stream), s)))
        return rc;
    return ok();
}

int softmax_matmul(const void *X, const void *Y, void *Z, int64_t M, int64_t K, int64_t N, void *stream)
{
    int rc;
    if ((rc = check_smm_args(X, Y, Z, M, K, N)))
        return rc;
    if (M == 0)
        return ok();
    const Layout l = smm_layout(M, K, N);
    Scratch s;
    if ((rc = s.alloc(l.total, l, static_cast<hipStream_t>(stream))))
        return rc;
    return softmax_matmul_ws(X, Y, Z, M, K, N, GMLP_PATH_AUTO, s.ptr, l.total, stream);
}

} // extern "C"
