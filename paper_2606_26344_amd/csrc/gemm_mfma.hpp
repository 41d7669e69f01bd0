// MFMA GEMM kernels of the Gated MLP for gfx950 (CDNA4).
//
// One template computes   C[n, m] = sum_k act[n, k] * W[k, m]
// for row-major activations act [N, K] (K contiguous) and weights W [K, M]
// (M contiguous), i.e. the matmuls of the Gated MLP graph (Fig.
// fig:mlp-example, Section 4.2) with N = tokens.  Two instantiations matter:
//
//   * dual-B gate/up:  NW = 2 weights (Wg, Wu) share every staged tile of X
//     (the paper's fusion of independent matmuls into one loop nest,
//     Section 4.5), and the epilogue writes H = bf16(act(r G) * (r U))
//     straight from the fp32 accumulators (act = silu, swish_beta or
//     sigmoid; r = the row's RMSNorm scale if one is given, else 1: the
//     paper's reorder of the RMSNorm multiply past the matmul, Section 2);
//     G and U never leave registers.
//   * down:            NW = 1 (Wd), epilogue writes Y = bf16(H Wd).
//   * paired gate/up:  NW = 1; the two blocks of a pair stream one weight
//     each (Wg or Wu) over the whole of K, for the same column tile, and the
//     later of the two combines its accumulators with the other's into
//     H = bf16(act(r G) * (r U)), through the split-K exchange below.  Each
//     block reads 256-byte row segments of one weight, with no fp32 partial
//     sums of K halves to exchange.
//
// Data flow per k-step of BK:
//   global --(buffer_load ... lds, 16 B per lane, zero-filled out of range)-->
//   LDS (STAGES-deep ring; 16-byte chunks XOR-swizzled so that the fragment
//   reads below are free of bank conflicts) --> registers --> MFMA.
//
// Operand roles.  v_mfma_f32_32x32x16_bf16 needs both operands K-contiguous
// per lane.  The activations are stored K-contiguous and are read with
// ds_read_b128.  The weights are stored M-contiguous, so they are read with
// the gfx950 transposing LDS load ds_read_b64_tr_b16: each 16-lane group
// fetches a 4 (k) x 16 (m) block and each lane receives one column's 4 k
// values.  The transpose thus happens inside the LDS read, never as a pass
// over memory (the paper fuses the transpose its matmul instruction needs
// into the data movement, Sections 4.4-4.5).
//
// The weights are the MFMA "A" operand (rows m) and the tokens the "B"
// operand (columns n), so the accumulator of a lane holds, for one token,
// runs of 4 consecutive output columns: the result is produced already in
// the row-major [N, M] layout of H and Y and is stored as 8-byte rows
// without any transpose (the operand swap the paper derives for
// transpose(nc_matmul(a, b)), Section 4.5).
//
// Schedule.  A block is 4 or 8 waves (one or two per SIMD; with two, the
// waves of a SIMD share its matrix core, so one issues MFMAs while the other
// waits on LDS or a barrier); each wave holds its share of the tile's fp32
// accumulators (at most 256 registers per lane with one wave per SIMD, 128
// with two).  Fragments are double-buffered in VGPRs, and the instruction order inside
// each k16 step is pinned with scheduling-group barriers: every MFMA is
// followed by one LDS fragment read for the next step and, in the step that
// follows a pipeline barrier, by one DMA issue for a future k-tile, so the
// matrix pipe does not wait on LDS latency or on issuing loads.
#pragma once

#include <utility>

#include "common.hpp"
#include "tiling.hpp"

namespace gmlp {

struct GemmParams {
    const uint16_t *w0;  // [K, M] bf16, M contiguous (Wg, or Wd)
    const uint16_t *w1;  // [K, M] bf16 second weight (Wu) of the dual kernel
    const uint16_t *act; // [N, K] bf16, K contiguous (X, or H)
    uint16_t *out;       // [N, M] bf16 (H, or Y)
    float *partial;      // split-K partial sums, fp32, [split][tile of the launch][wave][piece][lane]
    uint32_t *counters;  // split-K arrival counter per output tile (zero on entry and exit)
    int M, N, K;
    int k_split; // K rows per split (a multiple of BK when splits > 1)
    int splits;
    int tiles_m, tiles_n;
    int group_m; // consecutive blocks sweep group_m column tiles before the next token tile
    // This launch computes tiles [tile_base, tile_base + tile_count) of the
    // block order of all tiles_m x tiles_n tiles (a plan can give the tiles
    // of a last, partial round of blocks to a split-K part of their own).
    int tile_base, tile_count;
    // A split-K launch may start with head_blocks blocks (a multiple of 8)
    // that each compute one whole tile over all of K: tiles [0, head_blocks)
    // of the block order, before its split tiles, so those start as soon as
    // CUs free up instead of after the last whole tile.
    int head_blocks;
    // Gate/up epilogue: activation (enum Activation), swish slope, and the
    // per-token RMSNorm scales [N] (nullptr: none).
    int activation;
    float beta;
    const float *rrms;
    // Store epilogue: per-token divisors [N] (nullptr: none).  Softmax+MatMul
    // divides its result rows by the softmax sums here.
    const float *rowdiv;
};

// Physical 16-byte chunk of logical chunk c in row k of a weight tile.  The
// XOR keeps the 4 rows x 4 chunks read by 32 lanes of one transposing load
// on distinct banks (and the 4 x 2 read by 16 lanes), for 64 or 32 banks.
template <int CPR, bool M16>
__device__ __forceinline__ int w_swizzle(int k)
{
    if constexpr (CPR >= 16 && M16) {
        // The 16x16x32 reads take rows k and k + 16 in one pass as well
        // (lane groups 0 and 1 read k groups 0 and 2): the rows with bit 4
        // set use four other XOR values.
        const int g = k & 3;
        if (k & 16)
            return g == 0 ? 2 : g == 1 ? 4 : g == 2 ? 8 : 14;
        return g == 0 ? 0 : g == 1 ? 6 : g == 2 ? 10 : 12;
    } else if constexpr (CPR >= 16) {
        const int g = k & 3;
        return g == 0 ? 0 : g == 1 ? 6 : g == 2 ? 10 : 12;
    } else {
        return (k & 3) << 1;
    }
}

// The accumulators of one 32 x 32 output block of a wave: one
// v_mfma_f32_32x32x16_bf16 accumulator, or four v_mfma_f32_16x16x32_bf16
// ones (subtile j: columns 16 (j & 1) .., tokens 16 (j >> 1) ..).  Piece j is
// the lane's accumulators 4j .. 4j+3: 4 consecutive output columns of one
// token, starting at column col(j) and token tok(j) of the block.
template <bool M16>
struct AccBlock;
template <>
struct AccBlock<false> {
    f32x16 v;
    __device__ float get(int r) const { return v[r]; }
    __device__ void set(int r, float x) { v[r] = x; }
    __device__ f32x4 piece(int j) const { return f32x4{v[4 * j], v[4 * j + 1], v[4 * j + 2], v[4 * j + 3]}; }
    __device__ void set_piece(int j, const f32x4 &x)
    {
        v[4 * j] = x[0];
        v[4 * j + 1] = x[1];
        v[4 * j + 2] = x[2];
        v[4 * j + 3] = x[3];
    }
    __device__ static int col(int j, int lane) { return 8 * j + 4 * (lane >> 5); }
    __device__ static int tok(int, int lane) { return lane & 31; }
};
template <>
struct AccBlock<true> {
    f32x4 v[4];
    __device__ float get(int r) const { return v[r >> 2][r & 3]; }
    __device__ void set(int r, float x) { v[r >> 2][r & 3] = x; }
    __device__ f32x4 piece(int j) const { return v[j]; }
    __device__ void set_piece(int j, const f32x4 &x) { v[j] = x; }
    __device__ static int col(int j, int lane) { return 16 * (j & 1) + 4 * (lane >> 4); }
    __device__ static int tok(int j, int lane) { return 16 * (j >> 1) + (lane & 15); }
};

// Physical chunk of logical chunk c in LDS row r of an activation tile
// (rows of 8 chunks): any 8, and any aligned 16, consecutive rows reading
// one logical chunk hit distinct banks.
__device__ __forceinline__ int x_swizzle(int r) { return (r ^ (r >> 3)) & 7; }

// Pin the instruction order of one k16 step: each MFMA is followed by one
// global (DMA) load and one LDS read, while any remain.
template <int N_MFMA, int N_DS, int N_VMEM>
__device__ __forceinline__ void interleave_step()
{
    constexpr int kMFMA = 0x008, kDSRead = 0x100, kVMEMRead = 0x020;
    [&]<int... I>(std::integer_sequence<int, I...>) __attribute__((always_inline)) {
        (
            [&] {
                __builtin_amdgcn_sched_group_barrier(kMFMA, 1, 0);
                if constexpr (I < N_VMEM)
                    __builtin_amdgcn_sched_group_barrier(kVMEMRead, 1, 0);
                if constexpr (I < N_DS)
                    __builtin_amdgcn_sched_group_barrier(kDSRead, 1, 0);
            }(),
            ...);
    }(std::make_integer_sequence<int, N_MFMA>{});
    if constexpr (N_DS > N_MFMA)
        __builtin_amdgcn_sched_group_barrier(kDSRead, N_DS - N_MFMA, 0);
    if constexpr (N_VMEM > N_MFMA)
        __builtin_amdgcn_sched_group_barrier(kVMEMRead, N_VMEM - N_MFMA, 0);
}

// Which split and tile of a launch block `block` computes.  Each XCD gets a
// contiguous range of the order; within it, consecutive blocks sweep
// group_m column tiles for one token tile, then the next token tile, so the
// blocks resident on one XCD share few distinct weight and activation strips
// in its L2.
__device__ __forceinline__ int gemm_split_of_block(const GemmParams &p, int block)
{
    return xcd_contiguous_id(block, p.tile_count * p.splits) / p.tile_count;
}

// Block-uniform wait before a block's first activation load (the fused
// kernel's down blocks wait there for their rows of H); true when the
// activations are ready.
struct GemmNoWait {
    __device__ bool operator()() const { return true; }
};

// One block's work of a GEMM launch: the output tile (or split-K piece of
// it) of launch block `block`.  stage_ptr(std::integral_constant<int, I>)
// gives the LDS buffer of pipeline stage I.
// SPLIT selects the split-K variant (several blocks per output tile, summed
// by the last one); without it p.splits must be 1.  STREAM_W loads the
// weights with the nontemporal policy, for plans with one token tile, where
// every weight element is read by exactly one block (measured: 5% faster at
// T = 128, slower wherever several token tiles re-read a weight tile).
// ACT_POLICY and OUT_POLICY are the cache policies of the activation loads
// and the output stores (kCoherent where another kernel's blocks on other
// XCDs write or read them while this kernel runs: the fused kernel's H).
// wait() runs before the first activation load; if it returns false the
// block's sums become NaN, so every output it feeds is NaN.  Returns the
// first output column of the tile if this block wrote it, else -1.
template <class S, int EPI, bool SPLIT, bool STREAM_W, int ACT_POLICY = 0, int OUT_POLICY = 0,
          class StagePtr, class Wait = GemmNoWait>
__device__ __forceinline__ int gemm_block(const GemmParams &p, int block, StagePtr stage_ptr,
                                          const Wait &wait = Wait{})
{
    __shared__ int s_last;
    constexpr int NW = S::NW, TM = S::TM, TN = S::TN, STAGES = S::STAGES;
    constexpr int NWAVES = S::NWAVES, KSTEPS = S::KSTEPS;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % S::WM, wn = wave / S::WM;

    // Block -> (split, tile), as gemm_split_of_block; the head blocks of a
    // split-K launch take whole tiles (split 0 of 1).
    const bool head = SPLIT && block < p.head_blocks;
    const int ntiles = p.tile_count; // split tiles of this launch
    const int id = head ? xcd_contiguous_id(block, p.head_blocks)
                        : xcd_contiguous_id(block - (SPLIT ? p.head_blocks : 0), ntiles * p.splits);
    const int split = head ? 0 : id / ntiles;
    const int local = head ? id : id - split * ntiles; // split tiles: counter and partial slot
    const int tile_id = head ? id : p.tile_base + local;
    const int per_group = p.group_m * p.tiles_n;
    const int group = tile_id / per_group;
    const int first_m = group * p.group_m;
    const int group_w = min(p.tiles_m - first_m, p.group_m);
    const int in_group = tile_id - group * per_group;
    const int tm = first_m + in_group % group_w;
    const int tn = in_group / group_w;
    const int tile = local;
    const int M = p.M, N = p.N, K = p.K;
    const int m0 = tm * S::BMW, n0 = tn * S::BN;
    // A pair's blocks each take the whole of K; split selects the weight.
    constexpr bool PAIR = EPI == EPI_GATE_PAIR;
    static_assert(!PAIR || (NW == 1 && SPLIT), "a pair is two blocks of one weight each");
    const int kb = PAIR ? 0 : split * p.k_split;
    const int ke = PAIR || head ? K : min(K, kb + p.k_split);
    const uint16_t *w_first = PAIR && split ? p.w1 : p.w0;
    const int nk = (ke - kb + S::BK - 1) / S::BK;
    const bool ragged_k = (ke - kb) % S::BK != 0; // last k-tile is partial

    // ---- staging addresses ---------------------------------------------------
    // Weight load i of this lane: row i*W_RPI + w_k, physical chunk lane %
    // W_CPR holding the logical chunk that the row's swizzle maps there.  The
    // swizzle depends on the row only through bits 0, 1 and 4; bits 0 and 1
    // are the same for every i, and bit 4 of w_k + i*W_RPI flips with bit 4
    // of i*W_RPI, so two voffsets serve all i and the row step goes into the
    // scalar offset.
    const int w_k = wave * S::W_LPR + lane / S::W_CPR;
    auto w_voff_of = [&](int row) __attribute__((always_inline)) {
        const int c = (lane % S::W_CPR) ^ w_swizzle<S::W_CPR, S::M16>(row);
        return m0 + c * 8 < M ? (uint32_t)(w_k * M + c * 8) * 2u : kOutOfRange;
    };
    const uint32_t w_voff = w_voff_of(w_k), w_voff_b4 = w_voff_of(w_k ^ 16);
    static_assert(S::W_RPI % 4 == 0 && S::W_RPI >= 4, "row bits 0, 1 fixed across loads");
    static_assert(S::W_RPI >= 16 || (16 % S::W_RPI == 0), "bit 4 of w_k + i*W_RPI is that of w_k xor i*W_RPI");
    const uint32_t w_soff_step = (uint32_t)S::W_RPI * (uint32_t)M * 2u;
    // Activation load i: LDS row x_r(i) (8 rows per wave load), physical
    // chunk lane % 8 holding chunk x_c of token x_t.  Tokens past N are
    // clamped to N-1: they only feed output rows that are never stored.
    uint32_t x_voff[S::X_LOADS];
    int x_kcol[S::X_LOADS];
#pragma unroll
    for (int i = 0; i < S::X_LOADS; ++i) {
        const int r = (i * NWAVES + wave) * 8 + (lane >> 3);
        const int cc = (lane & 7) ^ x_swizzle(r);
        const int t = r + (cc / S::X_CPT) * S::X_ROWS;
        const int c = cc % S::X_CPT;
        x_kcol[i] = c * 8;
        x_voff[i] = (uint32_t)((min(n0 + t, N - 1) - n0) * K + c * 8) * 2u;
    }

    // Issue the DMA of k-tile kt into stage buffer sbuf, without branches so
    // that the loads can be interleaved with MFMAs.  A partial last tile
    // gets per-lane k masks (rows of W and columns of act past the end of
    // the k range read as zeros); a tile past the end (kt >= nk) reads only
    // zeros into a buffer nobody reads again, which keeps the count of loads
    // in flight the same at every step.
    auto issue = [&](uint8_t *sbuf, int kt) __attribute__((always_inline)) {
        const int k0 = kb + kt * S::BK;
        const int krem = kt < nk ? ke - k0 : 0;
        const bool masked = ragged_k ? kt >= nk - 1 : kt >= nk;
        const __amdgpu_buffer_rsrc_t rx = make_rsrc(p.act + (size_t)n0 * K + k0);
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const __amdgpu_buffer_rsrc_t rw = make_rsrc((w == 0 ? w_first : p.w1) + (size_t)k0 * M + m0);
#pragma unroll
            for (int i = 0; i < S::W_LOADS; ++i) {
                const uint32_t v = (masked && i * S::W_RPI + w_k >= krem) ? kOutOfRange
                                   : ((i * S::W_RPI) & 16)                  ? w_voff_b4
                                                                            : w_voff;
                uint8_t *dst = sbuf + w * S::W_TILE_BYTES + (i * NWAVES + wave) * 1024;
                if constexpr (STREAM_W)
                    load16_to_lds_stream(rw, dst, v, (uint32_t)i * w_soff_step);
                else
                    load16_to_lds(rw, dst, v, (uint32_t)i * w_soff_step);
            }
        }
#pragma unroll
        for (int i = 0; i < S::X_LOADS; ++i) {
            const uint32_t v = (masked && x_kcol[i] >= krem) ? kOutOfRange : x_voff[i];
            uint8_t *dst = sbuf + NW * S::W_TILE_BYTES + (i * NWAVES + wave) * 1024;
            if constexpr (ACT_POLICY != 0)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, GMLP_LDS(dst), 16, v, 0, 0, ACT_POLICY);
            else
                load16_to_lds(rx, dst, v);
        }
    };

    // ---- fragment read offsets ---------------------------------------------
    // 32x32x16: weight (A) fragment of m-tile mi for k16 step kk: a
    // transposing read of k rows kk*16 + r_lane (+4 for elements 4..7) in
    // column chunk c; each 16-lane group reads 4 rows x 16 columns, the two
    // groups of a half-wave the two 16-column halves, the two half-waves k
    // rows 0..7 and 8..15.  16x16x32: the 16-column half sa of m-tile mi for
    // k32 step kk: the four 16-lane groups g read k rows 8 kg(g) .. +7 of the
    // same 16 columns, kg = 0, 2, 1, 3 for g = 0, 1, 2, 3 (any order of the
    // four k groups gives the same sums if A and B share it; this one keeps
    // the lanes l and l + 32 that the LDS serves together on neighbouring
    // chunks of a token row, as the 32x32x16 layout does).
    constexpr bool M16 = S::M16;
    constexpr int SUB = M16 ? 2 : 1; // 16-wide halves of a 32-wide block per fragment
    using A = AccBlock<M16>;
    const int kg = ((lane >> 4) & 1) << 1 | (lane >> 5); // k group of a 16x16x32 lane group
    const int r_lane = M16 ? 8 * kg + ((lane & 15) >> 2) : 8 * (lane >> 5) + ((lane & 15) >> 2);
    int a_off[TM][SUB];
#pragma unroll
    for (int mi = 0; mi < TM; ++mi)
#pragma unroll
        for (int sa = 0; sa < SUB; ++sa) {
            const int c = wm * TM * 4 + mi * 4 + 2 * (M16 ? sa : (lane >> 4) & 1) + ((lane & 3) >> 1);
            a_off[mi][sa] = r_lane * S::W_ROW_BYTES + ((c ^ w_swizzle<S::W_CPR, S::M16>(r_lane)) << 4) + (lane & 1) * 8;
        }
    // Token (B) fragment of n-tile ni (32x32x16): token t = wn*TN*32 + ni*32
    // + lane%32, logical chunk 2*kk + lane/32 of that token, i.e. LDS row
    // t % X_ROWS, combined chunk 2*kk + lane/32 + X_CPT * (t / X_ROWS); the
    // chunk bits of the byte address are XORed with 32*kk for step kk.
    // 16x16x32: half sb of n-tile ni, token t = wn*TN*32 + ni*32 + 16 sb +
    // lane%16, chunk 4*kk + kg (XOR 64*kk).
    int b_off[TN][SUB];
#pragma unroll
    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
        for (int sb = 0; sb < SUB; ++sb) {
            const int t = wn * TN * 32 + ni * 32 + (M16 ? 16 * sb + (lane & 15) : lane & 31);
            const int r = t % S::X_ROWS;
            const int cc = (M16 ? kg : lane >> 5) + S::X_CPT * (t / S::X_ROWS);
            b_off[ni][sb] = r * 128 + ((cc ^ x_swizzle(r)) << 4);
        }

    A acc[NW][TM][TN];
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int mi = 0; mi < TM; ++mi)
#pragma unroll
            for (int ni = 0; ni < TN; ++ni)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[w][mi][ni].set_piece(j, f32x4{});

    struct Frags {
        bf16x8 a[NW][TM][SUB];
        bf16x8 b[TN][SUB];
    };
    auto load_frags = [&](Frags &f, const uint8_t *sbuf, int kk) __attribute__((always_inline)) {
        const uint8_t *sx = sbuf + NW * S::W_TILE_BYTES;
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int mi = 0; mi < TM; ++mi)
#pragma unroll
                for (int sa = 0; sa < SUB; ++sa) {
                    const uint8_t *pa = sbuf + w * S::W_TILE_BYTES + kk * S::MFMA_K * S::W_ROW_BYTES + a_off[mi][sa];
                    i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (__attribute__((address_space(3))) i16x4 *)GMLP_LDS(pa));
                    i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (__attribute__((address_space(3))) i16x4 *)GMLP_LDS(pa + 4 * S::W_ROW_BYTES));
                    f.a[w][mi][sa] =
                        __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                }
#pragma unroll
        for (int ni = 0; ni < TN; ++ni)
#pragma unroll
            for (int sb = 0; sb < SUB; ++sb)
                f.b[ni][sb] = *(const bf16x8 *)(sx + (b_off[ni][sb] ^ (2 * S::MFMA_K * kk)));
    };
    auto mma = [&](const Frags &f) __attribute__((always_inline)) {
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int mi = 0; mi < TM; ++mi)
#pragma unroll
                for (int ni = 0; ni < TN; ++ni) {
                    if constexpr (M16) {
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            acc[w][mi][ni].v[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                f.a[w][mi][j & 1], f.b[ni][j >> 1], acc[w][mi][ni].v[j], 0, 0, 0);
                    } else {
                        acc[w][mi][ni].v = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[w][mi][0], f.b[ni][0],
                                                                                   acc[w][mi][ni].v, 0, 0, 0);
                    }
                }
    };
    // 16x16x32: the A fragments of a k32 step are double-buffered (read for
    // the next step among this step's MFMAs), the B fragments are not: each
    // B fragment is read again for the next step right after the last of
    // its 4 MFMAs (NW x TM x 2 of them), so the fragments take no more
    // registers than the 32x32x16 ones.
    struct FragA {
        bf16x8 a[NW][TM][SUB];
    };
    struct FragB {
        bf16x8 b[TN][SUB];
    };
    auto load_a = [&](FragA &f, const uint8_t *sbuf, int kk) __attribute__((always_inline)) {
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int mi = 0; mi < TM; ++mi)
#pragma unroll
                for (int sa = 0; sa < SUB; ++sa) {
                    const uint8_t *pa = sbuf + w * S::W_TILE_BYTES + kk * S::MFMA_K * S::W_ROW_BYTES + a_off[mi][sa];
                    i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (__attribute__((address_space(3))) i16x4 *)GMLP_LDS(pa));
                    i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (__attribute__((address_space(3))) i16x4 *)GMLP_LDS(pa + 4 * S::W_ROW_BYTES));
                    f.a[w][mi][sa] =
                        __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                }
    };
    auto load_b = [&](FragB &f, const uint8_t *sbuf, int kk, int ni, int sb) __attribute__((always_inline)) {
        f.b[ni][sb] = *(const bf16x8 *)(sbuf + NW * S::W_TILE_BYTES + (b_off[ni][sb] ^ (2 * S::MFMA_K * kk)));
    };
    auto load_a1 = [&](FragA &f, const uint8_t *sbuf, int kk, int q) __attribute__((always_inline)) {
        const int w = q / (TM * SUB), mi = q / SUB % TM, sa = q % SUB;
        const uint8_t *pa = sbuf + w * S::W_TILE_BYTES + kk * S::MFMA_K * S::W_ROW_BYTES + a_off[mi][sa];
        i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4 *)GMLP_LDS(pa));
        i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) i16x4 *)GMLP_LDS(pa + 4 * S::W_ROW_BYTES));
        f.a[w][mi][sa] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    };
    // The MFMAs of one k32 step, one group per 16-token B fragment: its
    // NW x TM x 2 MFMAs, then (A fragments spread over the groups) the next
    // step's A reads and that B fragment's next read.  A scheduling fence
    // after each group keeps every B read after the MFMAs that still need
    // the old fragment, so the two never occupy registers at once.
    auto mma_roll = [&](const FragA &fa, FragA &fa_next, FragB &fb, const uint8_t *nbuf, int nkk)
                        __attribute__((always_inline)) {
        constexpr int GROUPS = TN * SUB, AFRAGS = NW * TM * SUB;
        constexpr int APG = (AFRAGS + GROUPS - 1) / GROUPS; // A fragments read per group
        [&]<int... G>(std::integer_sequence<int, G...>) __attribute__((always_inline)) {
            (
                [&] {
                    constexpr int ni = G / SUB, sb = G % SUB;
                    if constexpr (M16)
#pragma unroll
                        for (int w = 0; w < NW; ++w)
#pragma unroll
                            for (int mi = 0; mi < TM; ++mi)
#pragma unroll
                                for (int sa = 0; sa < SUB; ++sa)
                                    acc[w][mi][ni].v[sa + 2 * sb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                        fa.a[w][mi][sa], fb.b[ni][sb], acc[w][mi][ni].v[sa + 2 * sb], 0, 0, 0);
#pragma unroll
                    for (int q = G * APG; q < (G + 1) * APG && q < AFRAGS; ++q)
                        load_a1(fa_next, nbuf, nkk, q);
                    load_b(fb, nbuf, nkk, ni, sb);
                    __builtin_amdgcn_sched_barrier(0);
                }(),
                ...);
        }(std::make_integer_sequence<int, GROUPS>{});
    };
    // A tile has landed in LDS (for every wave) once at most the STAGES - 2
    // tiles issued after it are in flight and all waves have passed a
    // barrier.  Every step issues exactly one tile (real or past the end),
    // so the count is the same at every step.
    auto wait_tile = [&]() __attribute__((always_inline)) {
        wait_vmcnt<(STAGES - 2) * S::LOADS_PER_STAGE>();
        wait_lgkm0();
        barrier_only();
    };

    // ---- pipelined main loop -------------------------------------------------
    // Stage buffer of tile kt is kt % STAGES.  Fragments are double-buffered
    // in registers: the reads for k16 step kk+1 are issued among the MFMAs of
    // step kk.  Before the last step of a tile, a barrier makes the next
    // tile visible and frees this tile's buffer; the DMA of tile kt + STAGES
    // into it and the next tile's first fragment reads are then issued among
    // the last step's MFMAs.
    static_assert(KSTEPS % 2 == 0, "k steps alternate between two fragment buffers");
    static_assert(!M16 || KSTEPS == 2, "16x16x32: two k32 steps per k-tile");
    Frags f0, f1;
    FragA fa0, fa1;
    FragB fb;
    const bool ready = wait();
    [&]<int... I>(std::integer_sequence<int, I...>) __attribute__((always_inline)) {
        (issue(stage_ptr(std::integral_constant<int, I>{}), I), ...);
    }(std::make_integer_sequence<int, STAGES - 1>{});
    wait_tile();
    issue(stage_ptr(std::integral_constant<int, STAGES - 1>{}), STAGES - 1);
    if constexpr (M16) {
        load_a(fa0, stage_ptr(std::integral_constant<int, 0>{}), 0);
#pragma unroll
        for (int ni = 0; ni < TN; ++ni)
#pragma unroll
            for (int sb = 0; sb < SUB; ++sb)
                load_b(fb, stage_ptr(std::integral_constant<int, 0>{}), 0, ni, sb);
    } else {
        load_frags(f0, stage_ptr(std::integral_constant<int, 0>{}), 0);
    }

    // One k-tile held in stage buffer I, without branches: the registers
    // flow straight through (accumulators and fragments need no copies) and
    // each k step is one scheduling region.  At the last tile the next-tile
    // fragment read touches stale LDS and is unused.
    auto step = [&](auto stage, int kt) __attribute__((always_inline)) {
        constexpr int I = decltype(stage)::value;
        uint8_t *buf = stage_ptr(stage);
        uint8_t *next = stage_ptr(std::integral_constant<int, (I + 1) % STAGES>{});
        if constexpr (M16) {
            mma_roll(fa0, fa1, fb, buf, 1);
            wait_tile();
            issue(buf, kt + STAGES);
            mma_roll(fa1, fa0, fb, next, 0);
        } else {
            [&]<int... KK>(std::integer_sequence<int, KK...>) __attribute__((always_inline)) {
                (
                    [&] {
                        // k step KK: fragments of step KK+1 among its MFMAs.
                        if constexpr (KK % 2 == 0) {
                            load_frags(f1, buf, KK + 1);
                            mma(f0);
                        } else {
                            load_frags(f0, buf, KK + 1);
                            mma(f1);
                        }
                        interleave_step<S::MFMAS, S::FRAG_READS, 0>();
                    }(),
                    ...);
            }(std::make_integer_sequence<int, KSTEPS - 1>{});
            wait_tile();
            issue(buf, kt + STAGES);
            load_frags(f0, next, 0);
            mma(f1);
            interleave_step<S::MFMAS, S::FRAG_READS, S::LOADS_PER_STAGE>();
        }
    };
    int kt = 0;
    for (; kt + STAGES <= nk; kt += STAGES) {
        [&]<int... I>(std::integer_sequence<int, I...>) __attribute__((always_inline)) {
            (step(std::integral_constant<int, I>{}, kt + I), ...);
        }(std::make_integer_sequence<int, STAGES>{});
    }
    [&]<int... I>(std::integer_sequence<int, I...>) __attribute__((always_inline)) {
        ((kt + I < nk ? step(std::integral_constant<int, I>{}, kt + I) : void()), ...);
    }(std::make_integer_sequence<int, STAGES - 1>{});
    // Drain the loads issued past the end before LDS can be handed to
    // another block.
    wait_vmcnt<0>();
    if (!ready)
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
            for (int mi = 0; mi < TM; ++mi)
#pragma unroll
                for (int ni = 0; ni < TN; ++ni)
#pragma unroll
                    for (int e = 0; e < 16; ++e)
                        acc[w][mi][ni].set(e, __builtin_nanf(""));

    // ---- split-K: fixed-order reduction by the last block of each tile ----------
    // Each wave's partial sums go out as 16-byte device-coherent stores (sc1:
    // written through to memory, past the XCD-private L2) in a wave-contiguous
    // layout, [split][tile][wave][piece][lane], so every store instruction
    // writes 1 KB of consecutive bytes.  After they complete (vmcnt 0) the
    // block counts itself in; the last block of the tile reads each split's
    // pieces with device-coherent loads (up to 16 pieces of a split in flight
    // at once) and adds the splits in order 0, 1, 2, ...  No cache-wide
    // write-back or invalidate is needed.
    if (SPLIT && p.splits > 1 && !head) {
        constexpr int PIECES = NW * TM * TN * 4; // 4 accumulators (16 bytes) per piece
        const __amdgpu_buffer_rsrc_t prs = make_rsrc(p.partial);
        const uint32_t lane_off = lane * 16;
        auto wave_base = [&](int sp) __attribute__((always_inline)) {
            return (uint32_t)(((sp * ntiles + tile) * NWAVES + wave) * PIECES) * 1024u;
        };
        {
            const uint32_t base = wave_base(split);
#pragma unroll
            for (int w = 0; w < NW; ++w)
#pragma unroll
                for (int mi = 0; mi < TM; ++mi)
#pragma unroll
                    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const int g = ((w * TM + mi) * TN + ni) * 4 + j;
                            const f32x4 v = acc[w][mi][ni].piece(j);
                            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), prs, lane_off,
                                                                   base + g * 1024u, kCoherent);
                        }
        }
        wait_vmcnt<0>();
        __syncthreads();
        if (tid == 0) {
            const uint32_t before =
                __hip_atomic_fetch_add(p.counters + tile, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_last = before == (uint32_t)(p.splits - 1);
        }
        __syncthreads();
        if (!s_last)
            return -1;
        if (tid == 0)
            __hip_atomic_store(p.counters + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if constexpr (PAIR) {
            // This block's accumulators are G (split 0) or U (split 1); the
            // other block's are read back piece by piece, and every piece
            // gives 4 columns of H at once.
            static_assert(PIECES <= 24, "the other block's pieces are read in one pass");
            const uint32_t obase = wave_base(1 - split);
            f32x4 other[PIECES];
#pragma unroll
            for (int g = 0; g < PIECES; ++g)
                other[g] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(prs, lane_off,
                                                                                          obase + g * 1024u,
                                                                                          kCoherent));
            float rs[TN][SUB];
#pragma unroll
            for (int ni = 0; ni < TN; ++ni)
#pragma unroll
                for (int h = 0; h < SUB; ++h) {
                    const int t = n0 + wn * TN * 32 + ni * 32 + A::tok(2 * h, lane);
                    rs[ni][h] = p.rrms && t < N ? p.rrms[t] : 1.0f;
                }
            const __amdgpu_buffer_rsrc_t ro = make_rsrc(p.out + (size_t)n0 * M + m0);
#pragma unroll
            for (int g = 0; g < PIECES; ++g) {
                const int mi = g / (4 * TN) % TM, ni = g / 4 % TN, j = g % 4;
                const int fl = wm * TM * 32 + mi * 32 + A::col(j, lane);
                const int tl = wn * TN * 32 + ni * 32 + A::tok(j, lane);
                const float r = rs[ni][M16 ? j >> 1 : 0];
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float own = acc[0][mi][ni].get(4 * j + e);
                    float gv = split == 0 ? own : other[g][e], uv = split == 0 ? other[g][e] : own;
                    if (p.rrms) {
                        gv *= r;
                        uv *= r;
                    }
                    v[e] = gate_act(gv, p.activation, p.beta) * uv;
                }
                const uint32_t off = n0 + tl < N && m0 + fl < M ? (uint32_t)(tl * M + fl) * 2u : kOutOfRange;
                __builtin_amdgcn_raw_buffer_store_b64(u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])}, ro,
                                                      off, 0, OUT_POLICY);
            }
            return m0;
        }
        if constexpr (NW == 1 && PIECES > 16) {
            // Large store tiles: the last block reads its own partial sums
            // back as well, so the accumulators are dead once stored, and
            // sums each pass of CH pieces over the splits (in order 0, 1,
            // 2, ...: the same sums as below, its own pieces being the bits
            // it stored) and stores that pass's outputs before the next.
            // Keeping the accumulators live through the reduction and the
            // epilogue spilled registers.
            constexpr int CH = PIECES % 8 == 0 ? 8 : 4;
            static_assert(PIECES % CH == 0, "whole passes");
            const __amdgpu_buffer_rsrc_t ro = make_rsrc(p.out + (size_t)n0 * M + m0);
#pragma unroll
            for (int c0 = 0; c0 < PIECES; c0 += CH) {
                f32x4 sum[CH];
                for (int sp = 0; sp < p.splits; ++sp) {
                    const uint32_t base = wave_base(sp);
                    f32x4 x[CH];
#pragma unroll
                    for (int g = 0; g < CH; ++g)
                        x[g] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                             prs, lane_off, base + (c0 + g) * 1024u, kCoherent));
#pragma unroll
                    for (int g = 0; g < CH; ++g)
                        sum[g] = sp == 0 ? x[g] : sum[g] + x[g];
                }
#pragma unroll
                for (int g = 0; g < CH; ++g) {
                    // Piece c0 + g is piece j of acc[0][mi][ni].
                    const int mi = (c0 + g) / (4 * TN) % TM, ni = (c0 + g) / 4 % TN, j = (c0 + g) % 4;
                    const int fl = wm * TM * 32 + mi * 32 + A::col(j, lane);
                    const int tl = wn * TN * 32 + ni * 32 + A::tok(j, lane);
                    float v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        v[e] = sum[g][e];
                        if (EPI == EPI_STORE && p.rowdiv)
                            v[e] = v[e] / (n0 + tl < N ? p.rowdiv[n0 + tl] : 1.0f);
                    }
                    const uint32_t off = n0 + tl < N && m0 + fl < M ? (uint32_t)(tl * M + fl) * 2u : kOutOfRange;
                    __builtin_amdgcn_raw_buffer_store_b64(u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])}, ro,
                                                          off, 0, OUT_POLICY);
                }
            }
            return m0;
        }
        // Pieces are summed CH at a time: all of them for up to 16; the
        // 256 x 256 tiles take four passes of 8 (tiles of 20 pieces five
        // of 4), which keeps the loaded pieces and the sums within the
        // register budget next to the accumulators.  Piece g = ((w * TM + mi) * TN + ni) * 4 + j holds
        // accumulators 4j .. 4j+3 of acc[w][mi][ni].
        constexpr int CH = PIECES <= 16 ? PIECES : PIECES % 8 == 0 ? 8 : 4;
        static_assert(PIECES % CH == 0, "whole passes");
        auto get_piece = [&](int g) __attribute__((always_inline)) {
            return acc[g / (4 * TN * TM)][g / (4 * TN) % TM][g / 4 % TN].piece(g % 4);
        };
        auto set_piece = [&](int g, const f32x4 &v) __attribute__((always_inline)) {
            acc[g / (4 * TN * TM)][g / (4 * TN) % TM][g / 4 % TN].set_piece(g % 4, v);
        };
#pragma unroll
        for (int c0 = 0; c0 < PIECES; c0 += CH) {
            f32x4 sum[CH];
            for (int sp = 0; sp < p.splits; ++sp) {
                f32x4 x[CH];
                if (sp == split) {
#pragma unroll
                    for (int g = 0; g < CH; ++g)
                        x[g] = get_piece(c0 + g);
                } else {
                    const uint32_t base = wave_base(sp);
#pragma unroll
                    for (int g = 0; g < CH; ++g)
                        x[g] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                             prs, lane_off, base + (c0 + g) * 1024u, kCoherent));
                }
#pragma unroll
                for (int g = 0; g < CH; ++g)
                    sum[g] = sp == 0 ? x[g] : sum[g] + x[g];
            }
#pragma unroll
            for (int g = 0; g < CH; ++g)
                set_piece(c0 + g, sum[g]);
        }
    }

    // ---- epilogue: fp32 -> act(r G) * (r U), or acc / d -> bf16, 8-byte row-major stores --
    // Per-token scales of the lane's tokens: one per n-tile, or one per
    // 16-token half with the 16x16 subtiles.
    float rs[TN][SUB], ds[TN][SUB];
#pragma unroll
    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
        for (int h = 0; h < SUB; ++h) {
            const int t = n0 + wn * TN * 32 + ni * 32 + A::tok(2 * h, lane);
            rs[ni][h] = EPI == EPI_GATE_MUL && p.rrms && t < N ? p.rrms[t] : 1.0f;
            ds[ni][h] = EPI == EPI_STORE && p.rowdiv && t < N ? p.rowdiv[t] : 1.0f;
        }
    const bool scaled = EPI == EPI_GATE_MUL && p.rrms;
    const bool divided = EPI == EPI_STORE && p.rowdiv;
    // All of the wave's packed results first, each group of 4 columns into
    // registers of its own, then the stores back to back: a store's data
    // registers are not overwritten while it is in flight, so no store waits
    // for an earlier one to complete.
    u32x2 packed[TM][TN][4];
#pragma unroll
    for (int mi = 0; mi < TM; ++mi)
#pragma unroll
        for (int ni = 0; ni < TN; ++ni)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int h = M16 ? j >> 1 : 0;
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if constexpr (EPI == EPI_GATE_MUL) {
                        float g = acc[0][mi][ni].get(4 * j + e), u = acc[NW - 1][mi][ni].get(4 * j + e);
                        if (scaled) {
                            g *= rs[ni][h];
                            u *= rs[ni][h];
                        }
                        v[e] = gate_act(g, p.activation, p.beta) * u;
                    } else {
                        v[e] = acc[0][mi][ni].get(4 * j + e);
                        if (divided)
                            v[e] = v[e] / ds[ni][h];
                    }
                }
                packed[mi][ni][j] = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                // Keep the scheduler from pulling every accumulator out of
                // the AGPRs at once.
                __builtin_amdgcn_sched_barrier(0);
            }
    // Unconditional buffer stores relative to the tile's corner: a lane
    // whose element lies outside [N, M] stores at an offset past the buffer
    // range, which the hardware drops.  The largest in-range offset,
    // ((BN - 1) M + M - 4) * 2 bytes, stays below 2^31 for M <= 2^22.
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(p.out + (size_t)n0 * M + m0);
#pragma unroll
    for (int mi = 0; mi < TM; ++mi)
#pragma unroll
        for (int ni = 0; ni < TN; ++ni)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int fl = wm * TM * 32 + mi * 32 + A::col(j, lane);
                const int tl = wn * TN * 32 + ni * 32 + A::tok(j, lane);
                const uint32_t off = n0 + tl < N && m0 + fl < M ? (uint32_t)(tl * M + fl) * 2u : kOutOfRange;
                __builtin_amdgcn_raw_buffer_store_b64(packed[mi][ni][j], ro, off, 0, OUT_POLICY);
            }
    return m0;
}

template <class S, int EPI, bool SPLIT, bool STREAM_W>
__global__ __launch_bounds__(S::NTHREADS, 1) void gemm_mfma_kernel(GemmParams p)
{
    constexpr int STAGES = S::STAGES;
    // One LDS array per pipeline stage: distinct objects let the compiler see
    // that reading one stage does not depend on the DMA into another.
    __shared__ __attribute__((aligned(1024))) uint8_t lds0[S::STAGE_BYTES];
    __shared__ __attribute__((aligned(1024))) uint8_t lds1[S::STAGE_BYTES];
    __shared__ __attribute__((aligned(1024))) uint8_t lds2[STAGES > 2 ? S::STAGE_BYTES : 16];
    __shared__ __attribute__((aligned(1024))) uint8_t lds3[STAGES > 3 ? S::STAGE_BYTES : 16];
    __shared__ __attribute__((aligned(1024))) uint8_t lds4[STAGES > 4 ? S::STAGE_BYTES : 16];
    __shared__ __attribute__((aligned(1024))) uint8_t lds5[STAGES > 5 ? S::STAGE_BYTES : 16];
    __shared__ __attribute__((aligned(1024))) uint8_t lds6[STAGES > 6 ? S::STAGE_BYTES : 16];
    __shared__ __attribute__((aligned(1024))) uint8_t lds7[STAGES > 7 ? S::STAGE_BYTES : 16];
    auto stage_ptr = [&](auto s) __attribute__((always_inline)) -> uint8_t * {
        if constexpr (decltype(s)::value == 0) return lds0;
        else if constexpr (decltype(s)::value == 1) return lds1;
        else if constexpr (decltype(s)::value == 2) return lds2;
        else if constexpr (decltype(s)::value == 3) return lds3;
        else if constexpr (decltype(s)::value == 4) return lds4;
        else if constexpr (decltype(s)::value == 5) return lds5;
        else if constexpr (decltype(s)::value == 6) return lds6;
        else return lds7;
    };
    gemm_block<S, EPI, SPLIT, STREAM_W>(p, blockIdx.x, stage_ptr);
}

} // namespace gmlp
