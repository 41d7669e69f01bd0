// Host-side planning of libgmlp.so (csrc/plan.hpp) run on the host alone, for
// a build with AddressSanitizer and UndefinedBehaviorSanitizer: every path's
// plan, describe text and workspace layout over a grid of shapes up to the
// validated limits, argument validation with bad inputs, and the
// Softmax+MatMul plan.  Checks the plans' invariants as it goes and exits
// non-zero on the first violation (a sanitizer report aborts the run).
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "plan.hpp"

using namespace gmlp;

static int failures = 0;

#define EXPECT(cond, ...)                                                   \
    do {                                                                    \
        if (!(cond)) {                                                      \
            std::fprintf(stderr, "FAILED %s:%d: %s: ", __FILE__, __LINE__, #cond); \
            std::fprintf(stderr, __VA_ARGS__);                              \
            std::fprintf(stderr, "\n");                                     \
            if (++failures > 20)                                            \
                std::exit(1);                                               \
        }                                                                   \
    } while (0)

// A step covers its K range with its splits and its output with its tiles.
static void check_step(const Step &s, const Layout &l, int64_t T, int64_t D, int64_t F)
{
    EXPECT(s.kind != K_NONE, "T=%lld D=%lld F=%lld", (long long)T, (long long)D, (long long)F);
    EXPECT(s.blocks > 0 && s.threads > 0, "blocks %d threads %d", s.blocks, s.threads);
    EXPECT(s.splits >= 1 && s.k_split > 0, "splits %d k_split %d", s.splits, s.k_split);
    if (s.kind == K_GEMM_GU_P) // both blocks of a pair take the whole of K
        EXPECT(s.splits == 2 && s.k_split == s.K && s.tiles_n == 1, "pair of %d x %d vs K %d", s.splits,
               s.k_split, s.K);
    else
        EXPECT((int64_t)s.splits * s.k_split >= s.K && (int64_t)(s.splits - 1) * s.k_split < s.K,
               "splits %d x %d vs K %d", s.splits, s.k_split, s.K);
    EXPECT(s.partial_bytes <= l.rrms_off - l.partial_off, "partials %zu > %zu", s.partial_bytes,
           l.rrms_off - l.partial_off);
    EXPECT((size_t)s.counters * sizeof(uint32_t) <= kStripCounterBytes, "counters %d", s.counters);
    if (s.kind == K_GEMV) {
        EXPECT(s.strips * 8 * s.strip_lanes >= s.M, "strips %d", s.strips);
        EXPECT(s.counter_stride == 1 || s.counter_stride == kCounterLine, "counter stride %d", s.counter_stride);
        EXPECT(s.counters == (s.splits > 1 ? s.strips * s.counter_stride : 0), "GEMV counters %d", s.counters);
        EXPECT(s.blocks == s.strips * s.splits, "GEMV grid");
    } else {
        EXPECT((int64_t)s.tile_count + s.tail_tiles == (int64_t)s.tiles_m * s.tiles_n, "tiles %d + %d",
               s.tile_count, s.tail_tiles);
        EXPECT(s.blocks == s.tile_count * s.splits, "GEMM grid");
        if (s.tail_tiles) {
            const Step t = tail_step(s);
            EXPECT(t.splits >= 2 && t.splits <= kMaxTailSplits, "tail splits %d", t.splits);
            EXPECT((int64_t)t.splits * t.k_split >= t.K, "tail covers K");
            EXPECT(t.partial_bytes <= l.rrms_off - l.partial_off, "tail partials");
        }
    }
    EXPECT(!describe_step(s, true).empty(), "describe");
}

int main()
{
    const std::vector<int64_t> Ts = {1, 2, 3, 5, 6, 7, 8, 9, 15, 16, 17, 31, 32, 33, 48, 63, 64, 65,
                                     80, 96, 97, 100, 127, 128, 129, 200, 255, 256, 257, 300, 384, 511, 512, 640,
                                     520, 600, 768, 1000, 1024, 1088, 1280, 1536, 1600, 2048, 4096, 4352, 37601,
                                     1 << 20, 1 << 24};
    const std::vector<int64_t> dims = {8, 72, 136, 256, 264, 520, 1032, 2056, 4096, 4104, 4352, 8192,
                                       14336, 14464, 28672, 1 << 16, 1 << 22};
    int plans = 0;
    for (int64_t T : Ts)
        for (int64_t D : dims)
            for (int64_t F : dims) {
                if (check_shape(T, D, F) != GMLP_OK)
                    continue;
                const Layout l = make_layout(T, D, F);
                EXPECT(l.total >= l.rrms_off && l.rrms_off >= l.partial_off && l.partial_off >= l.h_off &&
                           l.h_off >= kCounterBytes,
                       "layout of T=%lld D=%lld F=%lld", (long long)T, (long long)D, (long long)F);
                EXPECT(l.partial_off - l.h_off >= (size_t)T * F * 2, "H fits");
                for (int path : {GMLP_PATH_AUTO, GMLP_PATH_GEMV, GMLP_PATH_MFMA, GMLP_PATH_FUSED,
                                 GMLP_PATH_FUSED_MFMA}) {
                    if (check_path(path, T) != GMLP_OK)
                        continue;
                    const Plan p = make_plan(T, D, F, path);
                    check_step(p.gate_up, l, T, D, F);
                    check_step(p.down, l, T, D, F);
                    if (p.rest_row) { // a token split of the gate/up step
                        check_step(p.gate_up_rest, l, T, D, F);
                        EXPECT(p.rest_row > 0 && p.rest_row < T && p.gate_up.N == p.rest_row &&
                                   p.gate_up_rest.N == T - p.rest_row && p.gate_up.M == F && p.gate_up_rest.M == F,
                               "token split of T=%lld at %lld", (long long)T, (long long)p.rest_row);
                    } else
                        EXPECT(p.gate_up.N == T, "gate/up rows");
                    if (p.path == GMLP_PATH_FUSED || p.path == GMLP_PATH_FUSED_MFMA)
                        EXPECT(fused_grid(p) == p.gate_up.blocks + p.down.blocks, "fused grid");
                    if (p.path == GMLP_PATH_FUSED_MFMA) {
                        // Both steps' counters and partial sums are live at once.
                        EXPECT(p.gate_up.tiles_n == 1 && p.down.tiles_n == 1, "one token tile");
                        // Where the counters fit (else the launch refuses the
                        // path), the layout holds both steps at once.
                        if (fused_mfma_counters_fit(p)) {
                            EXPECT(p.gate_up.tile_count + p.down.counters <= l.counters, "fused counters");
                            EXPECT(align_up(p.gate_up.partial_bytes) + p.down.partial_bytes <=
                                       l.rrms_off - l.partial_off,
                                   "fused partial sums");
                        }
                        EXPECT((size_t)l.counters * 4 <= kStripCounterBytes, "layout counters fit");
                        EXPECT(p.down.splits <= kFusedMaxSplits, "fused splits");
                        EXPECT(!fused_kernel_name(p).empty(), "fused name");
                    }
                    ++plans;
                }
                // Softmax+MatMul with M = T, K = F, N = D.
                if (check_smm_shape(T, F, D) == GMLP_OK) {
                    const Layout sl = smm_layout(T, F, D);
                    for (int path : {GMLP_PATH_AUTO, GMLP_PATH_MFMA})
                        check_step(smm_matmul_step(T, F, D, path), sl, T, D, F);
                }
            }
    EXPECT(plans > 1000, "only %d plans", plans);

    // Validation: rejected shapes and arguments never reach planning.
    const char *A = reinterpret_cast<const char *>(uintptr_t(1) << 40);
    const int64_t G = int64_t(1) << 34;
    EXPECT(validate(4, 256, 512, A, A + G, A + 2 * G, A + 3 * G, const_cast<char *>(A + 4 * G)) == GMLP_OK, "ok");
    EXPECT(validate(-1, 256, 512, A, A + G, A + 2 * G, A + 3 * G, A + 4 * G) == GMLP_ERR_INVALID_ARG, "T<0");
    EXPECT(validate(4, 260, 512, A, A + G, A + 2 * G, A + 3 * G, A + 4 * G) == GMLP_ERR_UNSUPPORTED, "D%%8");
    EXPECT(validate(4, 256, 512, A + 8, A + G, A + 2 * G, A + 3 * G, A + 4 * G) == GMLP_ERR_UNSUPPORTED, "align");
    EXPECT(validate(4, 256, 512, nullptr, A + G, A + 2 * G, A + 3 * G, A + 4 * G) == GMLP_ERR_INVALID_ARG, "null");
    EXPECT(validate(4, 256, 512, A, A + G, A + 2 * G, A + 3 * G, A + 16) == GMLP_ERR_INVALID_ARG, "alias");
    EXPECT(check_shape(int64_t(1) << 24, int64_t(1) << 22, 8) == GMLP_ERR_UNSUPPORTED,
           "a shape past the element limit");
    EXPECT(check_shape(8, int64_t(1) << 22, int64_t(1) << 22) == GMLP_ERR_UNSUPPORTED, "weights past the limit");
    EXPECT(check_shape((int64_t(1) << 24) + 1, 8, 8) == GMLP_ERR_UNSUPPORTED, "T past the limit");
    EXPECT(check_smm_shape(int64_t(1) << 24, int64_t(1) << 22, 8) == GMLP_ERR_UNSUPPORTED, "smm elements");
    EXPECT(check_shape(int64_t(1) << 62, 8, 8) == GMLP_ERR_UNSUPPORTED, "huge T");
    EXPECT(check_shape(8, int64_t(1) << 62, 8) == GMLP_ERR_UNSUPPORTED, "huge D");
    Variant v;
    EXPECT(check_variant(GMLP_ACT_SWISH, 1.702f, 1, 1e-6f, &v) == GMLP_OK && v.rms && v.beta == 1.702f, "variant");
    EXPECT(check_variant(7, 1.0f, 0, 0.0f, &v) == GMLP_ERR_INVALID_ARG, "activation");
    EXPECT(check_variant(GMLP_ACT_SWISH, __builtin_nanf(""), 0, 0.0f, &v) == GMLP_ERR_INVALID_ARG, "beta NaN");
    EXPECT(check_variant(GMLP_ACT_SILU, 1.0f, 1, -1.0f, &v) == GMLP_ERR_INVALID_ARG, "eps < 0");
    EXPECT(check_path(9, 4) == GMLP_ERR_INVALID_ARG && check_path(GMLP_PATH_GEMV, 9) == GMLP_ERR_UNSUPPORTED, "path");
    const Layout l = make_layout(16, 256, 512);
    EXPECT(check_workspace(nullptr, l.total, l) == GMLP_ERR_INVALID_ARG, "ws null");
    EXPECT(check_workspace(const_cast<char *>(A + 128), l.total, l) == GMLP_ERR_UNSUPPORTED, "ws align");
    EXPECT(check_workspace(const_cast<char *>(A), l.total - 1, l) == GMLP_ERR_NO_MEMORY, "ws size");
    // An error detail longer than its buffer is truncated, not overrun.
    std::string longname(2000, 'x');
    EXPECT(check_ptr(nullptr, longname.c_str(), true) == GMLP_ERR_INVALID_ARG && std::strlen(g_err) < sizeof g_err,
           "long detail");
    std::printf("host planning: %d plans checked, %d failures\n", plans, failures);
    return failures ? 1 : 0;
}
