/*
 * gmlp.h -- C ABI of the MI355X (gfx950) SiLU Gated MLP library, libgmlp.so.
 *
 * The operation (the paper's "SiLU Gated MLP" benchmark; graph in Fig.
 * fig:mlp-example, Section 4.1):
 *
 *     G = X Wg,   U = X Wu,   H = silu(G) * U,   Y = H Wd
 *
 * with matmul(a, b)[i, j] = sum_k a[i, k] b[k, j] (Fig. fig:op-sema,
 * Section 4.2.1) and silu(x) = x * sigmoid(x) (table tab:nki-ops,
 * Section 5.1).  W1, W2, W3 of the figure are Wg, Wu, Wd here.
 *
 * Numerics: every tensor is IEEE bfloat16 (bf16 bit patterns in uint16
 * storage).  Products are accumulated in fp32; G and U stay in fp32 registers;
 * silu is evaluated in fp32; H is rounded once to bf16 (round-to-nearest-even)
 * when it is written, and Y is rounded once to bf16 from its fp32 accumulator.
 *
 * Layout: all tensors are dense and row-major on the current HIP device:
 *     X  [T, D]     Wg [D, F]     Wu [D, F]     Wd [F, D]
 *     H  [T, F]     Y  [T, D]
 * T is the number of tokens (rows of X), D the model width, F the hidden
 * width.  D and F must be multiples of 8 and every pointer 16-byte aligned
 * (rows are then 16-byte aligned, which the kernels' 16-byte loads need).
 *
 * Ownership: the caller owns every tensor and every workspace; the library
 * never frees, keeps or reallocates caller memory, and holds no pointer after
 * a call returns.  Entry points without a workspace argument allocate their
 * scratch stream-ordered (hipMallocAsync/hipFreeAsync on the given stream).
 *
 * Streams: `stream` is a hipStream_t (NULL = the null stream).  Every compute
 * entry point only enqueues work and returns; kernel faults surface at the
 * caller's next synchronisation.  Calls on one stream are ordered; two calls
 * that share a workspace must not run concurrently (they would race on it).
 *
 * Errors: every entry point returns GMLP_OK (0) or a positive GMLP_ERR_*
 * code, never throws, and stores a human-readable detail for the calling
 * thread that gmlp_last_error() returns.  T == 0 is valid and launches
 * nothing.
 */
#ifndef GMLP_H
#define GMLP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GMLP_VERSION 100 /* 1.0.0 */

enum gmlp_status {
    GMLP_OK = 0,
    GMLP_ERR_INVALID_ARG = 1, /* null pointer, negative or overflowing size, aliasing output */
    GMLP_ERR_UNSUPPORTED = 2, /* D or F not a multiple of 8, misaligned pointer, size too large */
    GMLP_ERR_HIP = 3,         /* a HIP runtime call or kernel launch failed */
    GMLP_ERR_NO_MEMORY = 4,   /* scratch allocation failed, or workspace too small */
};

/* Which kernels compute the call (gmlp_forward_ex). */
enum gmlp_path {
    GMLP_PATH_AUTO = 0,  /* GEMV for T <= 5, MFMA GEMMs otherwise (measured faster from T = 6) */
    GMLP_PATH_GEMV = 1,  /* split-K streaming GEMV kernels; needs T <= 8 */
    GMLP_PATH_MFMA = 2,  /* MFMA GEMM kernels (any T) */
    GMLP_PATH_FUSED = 3, /* the whole MLP in one GEMV kernel: the first blocks run the gate/up
                            items, the rest the down items, each waiting only for the strips
                            of H its rows read; needs T <= 8; same Y as GMLP_PATH_GEMV bit for
                            bit.  Only for gmlp_forward_ex / gmlp_forward_variant.  The waits
                            are bounded (about a second): a down block that gives up makes the
                            strips of Y it feeds NaN and counts itself in the workspace's
                            give-up count (gmlp_workspace_status). */
    GMLP_PATH_FUSED_MFMA = 4, /* the two MFMA GEMMs of the few-token tiles in one kernel: the first
                                 blocks run the gate/up tiles, the rest the down tiles, each down
                                 block waiting only for the tiles of H its rows read (bounded
                                 waits as for GMLP_PATH_FUSED); needs T <= 64; same Y as the
                                 two-kernel GMLP_PATH_MFMA plan of the 32- and 64-token tiles, bit
                                 for bit.  Only for gmlp_forward_ex / gmlp_forward_variant. */
};

/*
 * Gate activations of the Gated MLP family, H = act(X Wg) * (X Wu).  The
 * paper benchmarks a SiLU and a SwiGLU Gated MLP and a GLU operator (Section
 * 6.1) without spelling them out; the usual definitions are used:
 */
enum gmlp_activation {
    GMLP_ACT_SILU = 0,    /* silu(g) = g * sigmoid(g)  (table tab:nki-ops, Section 5.1) */
    GMLP_ACT_SWISH = 1,   /* swish_beta(g) = g * sigmoid(beta * g)  (SwiGLU; beta = 1 is silu) */
    GMLP_ACT_SIGMOID = 2, /* sigmoid(g)  (GLU) */
};

/* Library version, GMLP_VERSION of the build. */
int gmlp_version(void);

/* Static name of a status code ("GMLP_OK", ...); never NULL. */
const char *gmlp_status_string(int status);

/* Detail of the last error returned to the calling thread ("" if none).
 * The string is owned by the library and valid until the thread's next call. */
const char *gmlp_last_error(void);

/*
 * Host-only check of the arguments of gmlp_forward: sizes (T >= 0, D > 0,
 * F > 0, D % 8 == 0, F % 8 == 0, D and F at most 2^22, T at most 2^24, and no
 * tensor of more than 2^37 elements: limits that keep the kernels' offsets
 * within a tile in 32 bits and every launch grid within range), non-NULL
 * 16-byte aligned pointers, and Y not overlapping any input.  Touches no
 * device memory and makes no HIP call.
 */
int gmlp_validate(int64_t T, int64_t D, int64_t F, const void *X, const void *Wg,
                  const void *Wu, const void *Wd, const void *Y);

/*
 * The kernels gmlp_forward_ex(..., path, ...) enqueues for this shape, as
 * text: one line per kernel, in launch order,
 *     "<kernel> grid=<blocks> block=<threads> k_splits=<n>\n"
 * with <kernel> as a profiler names it without the namespace (for example
 * "gemv_splitk_kernel<1, 2, 0, false>"), for the SiLU Gated MLP (the
 * variants of gmlp_forward_variant use the same plan; RMSNorm adds its
 * row-scale kernel on the MFMA path).  NUL-terminated, truncated to `bytes`
 * (which must be > 0).  Host-only: makes no HIP call.  Nothing for T == 0.
 * GMLP_OK, or INVALID_ARG / UNSUPPORTED for a bad shape, path or buffer.
 */
int gmlp_describe(int64_t T, int64_t D, int64_t F, int path, char *buf, size_t bytes);

/*
 * Bytes of workspace gmlp_forward_ws / gmlp_forward_ex need for this shape
 * (for any path).  The workspace holds H [T, F] bf16, fp32 split-K partial
 * sums and a block of arrival counters and barrier flags.  0 if the shape is
 * invalid.
 */
size_t gmlp_workspace_size(int64_t T, int64_t D, int64_t F);

/*
 * Prepare a workspace of `bytes` bytes for its first use: zero its counter
 * block (stream-ordered on `stream`).  The kernels return every counter to
 * zero when they finish, so this is needed once per fresh buffer, not per
 * call.  A buffer that was zero-filled by other means needs no init.
 */
int gmlp_workspace_init(void *workspace, size_t bytes, void *stream);

/*
 * Read and clear the give-up count of a workspace: the number of down blocks
 * of GMLP_PATH_FUSED and GMLP_PATH_FUSED_MFMA calls on it whose bounded wait
 * for H gave up since the last read (the parts of Y they feed were written
 * as NaN).  0 means every fused
 * call on the workspace completed normally.  Synchronises `stream` (the
 * stream the calls ran on) and copies 4 bytes to the host; not for use under
 * graph capture.  INVALID_ARG for a NULL pointer or `bytes` below the counter
 * block.
 */
int gmlp_workspace_status(void *workspace, size_t bytes, void *stream, uint32_t *fused_giveups);

/*
 * Test hook, not for production use: set how many times a down block of the
 * fused kernel polls for H before it gives up (default about a second of
 * polls) for the calls that follow, and return the previous value.  Tests
 * pass 0 to make the waits give up from the host, with every kernel still
 * running to completion.  Process-wide, not thread-safe against concurrent
 * fused calls.
 */
uint32_t gmlp_test_fused_spin_limit(uint32_t limit);

/*
 * Y = (silu(X Wg) * (X Wu)) Wd  for X [T, D], Wg/Wu [D, F], Wd [F, D],
 * Y [T, D], all bf16 device pointers (see the header comment for layout and
 * numerics).  Allocates its scratch stream-ordered on `stream`.
 */
int gmlp_forward(const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y,
                 int64_t T, int64_t D, int64_t F, void *stream);

/*
 * gmlp_forward with a caller-provided workspace of `ws_bytes` >=
 * gmlp_workspace_size(T, D, F) bytes, 256-byte aligned, prepared once with
 * gmlp_workspace_init.  Allocates nothing, issues no memset and leaves the
 * workspace's counters at zero, so a call can be captured in a HIP graph and
 * the graph replayed (the entry points that allocate their scratch cannot:
 * they allocate, clear and free per call).
 */
int gmlp_forward_ws(const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y,
                    int64_t T, int64_t D, int64_t F, void *workspace, size_t ws_bytes,
                    void *stream);

/*
 * gmlp_forward for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * kernels and results as gmlp_forward, bit for bit, with the workspace kept
 * in a static device array of GMLP_NOALLOC_SCRATCH_BYTES bytes inside the
 * library instead of memory allocated per call.  Makes no hipMalloc, hipFree
 * or other allocating call.  The caller still owns X, the weights and Y.
 *
 * Every device the library runs on holds one such array until the process
 * ends.  Its first call on a device takes the array's address and clears its
 * counters with a small kernel on `stream`; the kernels return the counters
 * to zero when they finish, so later calls find them zero.  All calls on one
 * device share that device's array and it keeps the last call's contents:
 * calls that overlap on one device (concurrent streams, host threads or
 * replayed graphs that are not ordered with each other) race on it and give
 * wrong results.  Order them on one stream, or use gmlp_forward_ws with a
 * workspace per stream.
 *
 * GMLP_ERR_UNSUPPORTED, with nothing launched, for a shape whose workspace
 * (gmlp_workspace_size) exceeds GMLP_NOALLOC_SCRATCH_BYTES (for example
 * T = 4096, D = 4096, F = 14336 needs 112 MiB); otherwise as gmlp_forward.
 */
#define GMLP_NOALLOC_SCRATCH_BYTES (64u << 20) /* 64 MiB per device */
int gmlp_forward_noalloc(const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y,
                         int64_t T, int64_t D, int64_t F, void *stream);

/* gmlp_forward_ws with the kernel path chosen explicitly (enum gmlp_path). */
int gmlp_forward_ex(const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y,
                    int64_t T, int64_t D, int64_t F, int path, void *workspace,
                    size_t ws_bytes, void *stream);

/*
 * A member of the Gated MLP family, with a caller workspace as for
 * gmlp_forward_ex:
 *     Y = (act(Xn Wg) * (Xn Wu)) Wd,
 * act = `activation` (enum gmlp_activation; `beta` is used by GMLP_ACT_SWISH
 * only and must be finite), and Xn = X, or with rmsnorm = 1 the RMSNorm of
 * X (the equation of Section 2, no gain): each row x becomes
 * x / sqrt(mean(x^2) + eps), eps finite and >= 0.  The normalisation is
 * never materialised: by the paper's reorder of the multiply past the
 * matmul, G and U are computed from X and scaled per row before act.  With
 * GMLP_ACT_SILU and rmsnorm = 0 this is gmlp_forward_ex, bit for bit.
 * INVALID_ARG for an unknown activation, a non-finite beta or a bad
 * rmsnorm/eps; otherwise as gmlp_forward_ex.
 */
int gmlp_forward_variant(const void *X, const void *Wg, const void *Wu, const void *Wd, void *Y,
                         int64_t T, int64_t D, int64_t F, int activation, float beta,
                         int rmsnorm, float eps, int path, void *workspace, size_t ws_bytes,
                         void *stream);

/*
 * First half of the graph alone (the paper's "MM+MM+SiLU+Mul" kernel):
 * H = bf16(silu(X Wg) * (X Wu)), H [T, F].  Allocates its scratch
 * stream-ordered on `stream`.
 */
int gmlp_gate_up(const void *X, const void *Wg, const void *Wu, void *H, int64_t T,
                 int64_t D, int64_t F, void *stream);

/* Down projection alone: Y = bf16(H Wd), H [T, F], Wd [F, D], Y [T, D].
 * Allocates its scratch stream-ordered on `stream`. */
int gmlp_down(const void *H, const void *Wd, void *Y, int64_t T, int64_t F, int64_t D,
              void *stream);

/*
 * gmlp_gate_up and gmlp_down with the kernel path chosen explicitly (enum
 * gmlp_path) and a caller-provided workspace sized by
 * gmlp_workspace_size(T, D, F) and prepared by gmlp_workspace_init (its H
 * region is not used: H is the caller's).  Allocate nothing; each enqueues
 * exactly one kernel.  gmlp_forward_ex gives the same bits as gmlp_gate_up_ws
 * into the workspace's H followed by gmlp_down_ws.
 */
int gmlp_gate_up_ws(const void *X, const void *Wg, const void *Wu, void *H, int64_t T,
                    int64_t D, int64_t F, int path, void *workspace, size_t ws_bytes,
                    void *stream);

/* The gate/up step of gmlp_forward_variant alone: H = bf16(act(Xn Wg) * (Xn Wu)),
 * with the same activation, beta, rmsnorm and eps arguments. */
int gmlp_gate_up_variant(const void *X, const void *Wg, const void *Wu, void *H, int64_t T,
                         int64_t D, int64_t F, int activation, float beta, int rmsnorm,
                         float eps, int path, void *workspace, size_t ws_bytes, void *stream);
int gmlp_down_ws(const void *H, const void *Wd, void *Y, int64_t T, int64_t F, int64_t D,
                 int path, void *workspace, size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* GMLP_H */
