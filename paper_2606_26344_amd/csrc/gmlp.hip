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
#include "gemm_fused.hpp"
#include "gemv.hpp"
#include "rmsnorm.hpp"
#include "softmax.hpp"
#include "plan.hpp"

using namespace gmlp;

namespace {

// Polls of a ready word (each with a short sleep) before a down block of the
// fused kernel stops waiting: about a second, far beyond any real wait.
// gmlp_test_fused_spin_limit changes it (tests force a give-up with 0).
constexpr uint32_t kSpinLimit = 1u << 20;
std::atomic<uint32_t> g_spin_limit{kSpinLimit};

int hip_check(hipError_t e, const char *what)
{
    if (e != hipSuccess)
        return fail(GMLP_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return GMLP_OK;
}

// ---- launches ----------------------------------------------------------------


GemmParams gemm_params(const Step &s, const void *w0, const void *w1, const void *act, void *out, uint8_t *ws,
                       const Layout &l, const Variant &v, const float *rrms, const float *rowdiv)
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
    p.head_blocks = 0;
    p.activation = v.act;
    p.beta = v.beta;
    p.rrms = rrms;
    p.rowdiv = rowdiv;
    return p;
}

template <class S, int EPI, bool SPLIT, bool STREAM_W = false>
int launch_gemm(const Step &s, const void *w0, const void *w1, const void *act, void *out,
                uint8_t *ws, const Layout &l, const Variant &v, const float *rrms, const float *rowdiv,
                hipStream_t stream, int head_blocks = 0)
{
    GemmParams p = gemm_params(s, w0, w1, act, out, ws, l, v, rrms, rowdiv);
    if (head_blocks && (!SPLIT || head_blocks % 8 != 0))
        return fail(GMLP_ERR_INVALID_ARG, "internal: %d whole-tile head blocks", head_blocks);
    p.head_blocks = head_blocks;
    if (!SPLIT && s.splits != 1)
        return fail(GMLP_ERR_INVALID_ARG, "internal: split-K plan for a kernel without split-K");
    if (s.partial_bytes > (size_t)kNumRecords)
        return fail(GMLP_ERR_UNSUPPORTED, "split-K partial sums of %zu bytes exceed the 2 GiB buffer range",
                    s.partial_bytes);
    hipLaunchKernelGGL((gemm_mfma_kernel<S, EPI, SPLIT, STREAM_W>), dim3(head_blocks + s.blocks), dim3(S::NTHREADS), 0,
                       stream, p);
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
    p.counter_stride = s.counter_stride;
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
    using L = GemvLayout<NT, NW>;
    if (s.threads != L::THREADS || s.strip_lanes != L::LANES)
        return fail(GMLP_ERR_INVALID_ARG, "internal: GEMV plan for %d threads and %d lanes, kernel of %d and %d",
                    s.threads, s.strip_lanes, L::THREADS, L::LANES);
    hipLaunchKernelGGL((gemv_splitk_kernel<NT, NW, EPI, RMS>), dim3(s.blocks), dim3(L::THREADS), 0,
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
// The MFMA path with RMSNorm: r = 1 / sqrt(mean(x^2) + eps) for every row of
// X [N, K] into the workspace, for the gate/up epilogue to scale G and U by.
int launch_row_rms(const Step &s, const void *X, uint8_t *ws, const Layout &l, const Variant &v,
                   hipStream_t st, const float **rrms)
{
    float *r = reinterpret_cast<float *>(ws + l.rrms_off);
    const int per = kRowRmsThreads / 64;
    hipLaunchKernelGGL(row_rms_kernel, dim3((unsigned)cdiv(s.N, per)), dim3(kRowRmsThreads), 0, st,
                       static_cast<const uint16_t *>(X), r, s.N, s.K, v.eps);
    *rrms = r;
    return hip_check(hipGetLastError(), "row RMS launch");
}

int run_gate_up(const Step &s, const void *X, const void *Wg, const void *Wu, void *H, uint8_t *ws,
                const Layout &l, const Variant &v, hipStream_t st)
{
    const float *rrms = nullptr;
    if (v.rms && s.kind != K_GEMV) {
        const int rc = launch_row_rms(s, X, ws, l, v, st, &rrms);
        if (rc)
            return rc;
    }
    switch (s.kind) {
    case K_GEMM_GU_L: {
        if (!s.tail_tiles)
            return launch_gemm<GateUpLarge, EPI_GATE_MUL, false>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
        return launch_gemm<GateUpLarge, EPI_GATE_MUL, true>(tail_step(s), Wg, Wu, X, H, ws, l, v, rrms, nullptr, st,
                                                            s.tile_count);
    }
    case K_GEMM_GU_S:
        return stream_weights(s) ? launch_gemm<GateUpSmall, EPI_GATE_MUL, true, true>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st)
                                 : launch_gemm<GateUpSmall, EPI_GATE_MUL, true, false>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
    case K_GEMM_GU_T: // one token tile: always streamed
        return launch_gemm<GateUpTiny, EPI_GATE_MUL, true, true>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
    case K_GEMM_GU_M:
        return stream_weights(s) ? launch_gemm<GateUpMid, EPI_GATE_MUL, true, true>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st)
                                 : launch_gemm<GateUpMid, EPI_GATE_MUL, true, false>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
    case K_GEMM_GU_Y:
        return launch_gemm<GateUp192, EPI_GATE_MUL, false>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
    case K_GEMM_GU_W: // one token tile: always streamed
        return launch_gemm<GateUpMid96, EPI_GATE_MUL, true, true>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
    case K_GEMM_GU_P: // one token tile, a G and a U block per column tile
        if (s.splits != 2 || s.tiles_n != 1)
            return fail(GMLP_ERR_INVALID_ARG, "internal: paired gate/up plan with %d splits, %d token tiles",
                        s.splits, s.tiles_n);
        if (s.N <= PairMid96::BN)
            return launch_gemm<PairMid96, EPI_GATE_PAIR, true, true>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
        if (s.N <= PairSmall::BN)
            return launch_gemm<PairSmall, EPI_GATE_PAIR, true, true>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
        if (s.N <= PairMid160::BN)
            return launch_gemm<PairMid160, EPI_GATE_PAIR, true, true>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
        return launch_gemm<PairMid192, EPI_GATE_PAIR, true, true>(s, Wg, Wu, X, H, ws, l, v, rrms, nullptr, st);
    case K_GEMV:
        return v.rms ? launch_gemv<2, EPI_GATE_MUL, true>(s, Wg, Wu, X, H, ws, l, v, st)
                     : launch_gemv<2, EPI_GATE_MUL, false>(s, Wg, Wu, X, H, ws, l, v, st);
    default: return fail(GMLP_ERR_INVALID_ARG, "no gate/up kernel for this plan");
    }
}

// The gate/up step of a plan: on a token split, the rest rows follow as a
// problem of their own, at offset rows of X and H.
int run_gate_up_plan(const Plan &p, const void *X, const void *Wg, const void *Wu, void *H, int64_t D,
                     int64_t F, uint8_t *ws, const Layout &l, const Variant &v, hipStream_t st)
{
    int rc = run_gate_up(p.gate_up, X, Wg, Wu, H, ws, l, v, st);
    if (rc || !p.rest_row)
        return rc;
    return run_gate_up(p.gate_up_rest, static_cast<const uint16_t *>(X) + p.rest_row * D, Wg, Wu,
                       static_cast<uint16_t *>(H) + p.rest_row * F, ws, l, v, st);
}

// The down step, Y = bf16(H Wd), or with row divisors d, Y = bf16((H Wd) / d)
// row by row (the divide of Softmax+MatMul moved past its matmul).
int run_down(const Step &s, const void *H, const void *Wd, void *Y, uint8_t *ws, const Layout &l,
             hipStream_t st, const float *rowdiv = nullptr)
{
    const Variant plain;
    switch (s.kind) {
    case K_GEMM_DN_L: {
        if (s.splits > 1)
            return launch_gemm<DownLarge, EPI_STORE, true>(s, Wd, nullptr, H, Y, ws, l, plain, nullptr, rowdiv, st);
        if (!s.tail_tiles)
            return launch_gemm<DownLarge, EPI_STORE, false>(s, Wd, nullptr, H, Y, ws, l, plain, nullptr, rowdiv, st);
        return launch_gemm<DownLarge, EPI_STORE, true>(tail_step(s), Wd, nullptr, H, Y, ws, l, plain, nullptr,
                                                        rowdiv, st, s.tile_count);
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
    case K_GEMM_DN_X:
        return launch_gemm<DownWide, EPI_STORE, true>(s, Wd, nullptr, H, Y, ws, l, plain, nullptr, rowdiv, st);
    case K_GEMM_DN_Q: // one token tile: always streamed
        return launch_gemm<DownMid160, EPI_STORE, true, true>(s, Wd, nullptr, H, Y, ws, l, plain, nullptr, rowdiv, st);
    case K_GEMM_DN_Y:
        return stream_weights(s) ? launch_gemm<DownMid192, EPI_STORE, true, true>(s, Wd, nullptr, H, Y, ws, l, plain,
                                                                                  nullptr, rowdiv, st)
                                 : launch_gemm<DownMid192, EPI_STORE, true, false>(s, Wd, nullptr, H, Y, ws, l, plain,
                                                                                   nullptr, rowdiv, st);
    case K_GEMM_DN_W: // one token tile: always streamed
        return launch_gemm<DownMid96, EPI_STORE, true, true>(s, Wd, nullptr, H, Y, ws, l, plain, nullptr, rowdiv, st);
    case K_GEMV: return launch_gemv<1, EPI_STORE, false>(s, Wd, nullptr, H, Y, ws, l, plain, st, rowdiv);
    default: return fail(GMLP_ERR_INVALID_ARG, "no down kernel for this plan");
    }
}


template <int NT, bool RMS>
int launch_fused_nt(const Plan &plan, const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y,
                    uint8_t *ws, const Layout &l, const Variant &v, hipStream_t st)
{
    if (plan.down.splits > kFusedMaxSplits)
        return fail(GMLP_ERR_UNSUPPORTED, "fused path: %d down splits, at most %d", plan.down.splits,
                    kFusedMaxSplits);
    if ((size_t)(plan.gate_up.strips + plan.down.strips) * plan.gate_up.counter_stride * sizeof(uint32_t) >
        kStripCounterBytes)
        return fail(GMLP_ERR_UNSUPPORTED, "fused path: too many strips for the counter block");
    void *H = ws + l.h_off;
    GemvFusedParams fp;
    fp.gate_up = gemv_params(plan.gate_up, Wg, Wu, X, H, ws, l, v, nullptr);
    fp.down = gemv_params(plan.down, Wd, nullptr, H, Y, ws, l, Variant{}, nullptr);
    fp.down.counters = fp.gate_up.counters + plan.gate_up.strips * plan.gate_up.counter_stride;
    fp.down.partial = reinterpret_cast<float *>(ws + l.partial_off + align_up(plan.gate_up.partial_bytes));
    fp.ready = reinterpret_cast<uint32_t *>(ws + l.counters_off + kStripCounterBytes);
    fp.errors = reinterpret_cast<uint32_t *>(ws + l.counters_off + kErrorOffset);
    fp.spin_limit = g_spin_limit.load();
    hipLaunchKernelGGL((gemv_fused_kernel<NT, RMS>), dim3(fused_grid(plan)), dim3(GemvLayout<NT, 2>::THREADS), 0,
                       st, fp);
    return hip_check(hipGetLastError(), "fused kernel launch");
}

// The one-launch MFMA path: gate/up tiles on the first blocks, down tiles on
// the rest (gemm_fused.hpp).  Both steps' split-K counters and partial sums
// are live at once: down's follow gate/up's.
int launch_fused_mfma(const Plan &plan, const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y,
                      uint8_t *ws, const Layout &l, const Variant &v, hipStream_t st)
{
    const Step &gu = plan.gate_up, &dn = plan.down;
    const bool tiny = gu.kind == K_GEMM_GU_T && dn.kind == K_GEMM_DN_T;
    const bool mid = gu.kind == K_GEMM_GU_M && dn.kind == K_GEMM_DN_M;
    if (!(tiny || mid) || gu.tiles_n != 1 || dn.tiles_n != 1)
        return fail(GMLP_ERR_INVALID_ARG, "internal: fused MFMA path needs the few-token tiles");
    if (dn.splits > kFusedMaxSplits)
        return fail(GMLP_ERR_UNSUPPORTED, "fused MFMA path: %d down splits, at most %d", dn.splits,
                    kFusedMaxSplits);
    if (!fused_mfma_counters_fit(plan))
        return fail(GMLP_ERR_UNSUPPORTED, "fused MFMA path: %d + %d tiles exceed the counter block", gu.tile_count,
                    dn.counters);
    if (align_up(gu.partial_bytes) + dn.partial_bytes > (size_t)kNumRecords)
        return fail(GMLP_ERR_UNSUPPORTED, "fused MFMA path: split-K partial sums exceed the 2 GiB buffer range");
    const float *rrms = nullptr;
    if (v.rms) {
        const int rc = launch_row_rms(gu, X, ws, l, v, st, &rrms);
        if (rc)
            return rc;
    }
    void *H = ws + l.h_off;
    GemmFusedParams fp;
    fp.gate_up = gemm_params(gu, Wg, Wu, X, H, ws, l, v, rrms, nullptr);
    fp.down = gemm_params(dn, Wd, nullptr, H, Y, ws, l, Variant{}, nullptr, nullptr);
    fp.down.counters = fp.gate_up.counters + gu.tile_count;
    fp.down.partial = reinterpret_cast<float *>(ws + l.partial_off + align_up(gu.partial_bytes));
    fp.ready = reinterpret_cast<uint32_t *>(ws + l.counters_off + kStripCounterBytes);
    fp.errors = reinterpret_cast<uint32_t *>(ws + l.counters_off + kErrorOffset);
    fp.spin_limit = g_spin_limit.load();
    const dim3 grid(fused_grid(plan));
    static_assert(FusedDownTiny::BMW == DownTiny::BMW && FusedDownTiny::BN == DownTiny::BN &&
                      FusedDownTiny::BK == DownTiny::BK && FusedDownMid::BMW == DownMid::BMW &&
                      FusedDownMid::BN == DownMid::BN && FusedDownMid::BK == DownMid::BK,
                  "the fused down steps run the planned tiles");
    if (tiny)
        hipLaunchKernelGGL((gemm_fused_kernel<GateUpTiny, FusedDownTiny>), grid, dim3(GateUpTiny::NTHREADS), 0, st,
                           fp);
    else
        hipLaunchKernelGGL((gemm_fused_kernel<GateUpMid, FusedDownMid>), grid, dim3(GateUpMid::NTHREADS), 0, st, fp);
    return hip_check(hipGetLastError(), "fused MFMA kernel launch");
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
    if (plan.path == GMLP_PATH_FUSED || plan.path == GMLP_PATH_FUSED_MFMA) {
        const std::string name = fused_kernel_name(plan);
        line(name.c_str(), fused_grid(plan), plan.gate_up.threads, plan.gate_up.splits);
        snprintf(buf, bytes, "%s", text.c_str());
        return ok();
    }
    text += describe_step(plan.gate_up, true);
    if (plan.rest_row)
        text += describe_step(plan.gate_up_rest, true);
    text += describe_step(plan.down, false);
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
    if (plan.path == GMLP_PATH_FUSED_MFMA) {
        rc = launch_fused_mfma(plan, X, Wg, Wu, Wd, Y, ws, l, v, st);
        return rc ? rc : ok();
    }
    void *H = ws + l.h_off;
    if ((rc = run_gate_up_plan(plan, X, Wg, Wu, H, D, F, ws, l, v, st)) ||
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
    if ((rc = run_gate_up_plan(plan, X, Wg, Wu, H, D, F, static_cast<uint8_t *>(workspace), l, v,
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
