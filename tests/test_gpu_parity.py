"""GPU parity: the HIP path (through the C ABI) against the CPU fp64 oracle.

Acceptance per output element: |Y_gpu - Y_ref| <= 1e-2 * (|Y_ref| + rms(Y_ref)),
rms over the checked elements, for bf16 inputs with fp32 accumulation.  The
same rule is applied to H for the gate/up step alone.  Shapes that the oracle
can finish in seconds are checked in full; the full-size workloads are
checked on sampled rows (rows are independent: the oracle computes exactly
those rows), in the same launch configuration the benchmark times.
"""
import numpy as np
import pytest
import torch

from paper_2606_26344_amd import gmlp
from paper_2606_26344_amd import inputs as I

pytestmark = pytest.mark.gpu

TOL = 1e-2


def _dev(bits):
    return gmlp.from_bf16_bits(bits)


def _check(got_bits, ref, what=""):
    got = I.bf16_bits_to_f32(got_bits).astype(np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), "non-finite output " + what
    rms = float(np.sqrt(np.mean(ref ** 2)))
    bound = TOL * (np.abs(ref) + rms)
    err = np.abs(got - ref)
    ratio = float(np.max(err / bound)) if err.size else 0.0
    print("%s max err/bound = %.3f (rms ref %.4g)" % (what, ratio, rms), flush=True)
    assert np.all(err <= bound), "%s: %d elements out of tolerance, worst ratio %.3f" % (
        what, int(np.sum(err > bound)), ratio)
    return ratio


def _run(T, D, F, seed=0, path="auto", rows=None, unit_rms=False, orc=None):
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=seed, unit_rms_rows=unit_rms)
    x, wg, wu, wd = (_dev(a) for a in (X, Wg, Wu, Wd))
    ws = gmlp.Workspace(T, D, F)
    y = gmlp.forward(x, wg, wu, wd, path=path, workspace=ws)
    torch.cuda.synchronize()
    Y = gmlp.to_bf16_bits(y)
    if rows is None:
        rows = np.arange(T)
    ref = orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows)
    return _check(Y[rows], ref, "T=%d D=%d F=%d path=%s" % (T, D, F, path))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    gmlp.library()  # fails loudly when libgmlp.so is missing


def test_tiny_workload(orc):
    w = I.WORKLOADS["tiny"]
    _run(w.T, w.D, w.F, seed=w.seed, orc=orc)


# Ragged shapes: T, D, F not multiples of the tile sizes (D, F multiples of
# 8), both paths and every tile configuration.
RAGGED = [
    (1, 256, 512), (2, 264, 520), (3, 520, 264), (4, 256, 1032), (5, 264, 264),
    (7, 256, 1032), (8, 264, 264), (9, 256, 512), (15, 264, 520), (16, 520, 1032),
    (17, 520, 1032), (33, 72, 136), (127, 256, 520), (128, 264, 1032), (129, 520, 264),
    (255, 256, 264), (257, 264, 520), (300, 1032, 2056),
    # 32-, 64- and 96-token tiles (T <= 32, T <= 64, T <= 96), at their edges.
    (32, 264, 1032), (48, 4104, 2056), (64, 520, 264), (65, 264, 520), (80, 1032, 264),
    (96, 264, 1032), (97, 520, 264),
]


@pytest.mark.parametrize("T,D,F", RAGGED, ids=["T%dD%dF%d" % s for s in RAGGED])
def test_ragged_shapes(orc, T, D, F):
    _run(T, D, F, seed=T + D + F, orc=orc)


def test_hidden_activations_past_2_gib(orc):
    """H [T, F] of more than 2 GiB (T = 37601, F = 28672: 2.008 GiB): tile
    base addresses are formed in 64 bits and only offsets within a tile are
    32-bit.  The checked rows include the last ones, which lie past 2 GiB in
    H, and rows of the down step's split-K tail tiles."""
    T, D, F = 37601, 4096, 28672
    assert T * F * 2 > 2 ** 31
    rows = np.array([0, 1, 18000, 37119, 37120, 37448, 37449, 37520, 37599, 37600])
    _run(T, D, F, seed=11, rows=rows, orc=orc)


def _random_shapes(n, seed):
    # Token counts over every plan (GEMV, 32/64/96/128-token tiles, two token
    # tiles, 256-token tiles), D and F multiples of 8 up to 2056.
    r = np.random.default_rng(seed)
    t_choices = [1, 2, 3, 4, 5, 6, 7, 8, 9, 31, 32, 33, 64, 65, 96, 97, 127, 128, 129, 200, 256, 257, 384, 600]
    return [(int(r.choice(t_choices)), 8 * int(r.integers(1, 258)), 8 * int(r.integers(1, 258)))
            for _ in range(n)]


RANDOM = _random_shapes(16, seed=2024)
WAIVER_CAP = 0.005  # largest fraction of elements judged against Yb only


@pytest.mark.parametrize("T,D,F", RANDOM, ids=["T%dD%dF%d" % s for s in RANDOM])
def test_random_shapes(orc, T, D, F):
    # Two references from the oracle: the plain definition Y (fp64 H), and
    # Yb, the same with H rounded once to bf16 as the library's stated
    # numerics prescribe (the oracle's own fp64 H, rounded here, then the
    # oracle's down step).  With few hidden columns that rounding alone can
    # take an output past the tolerance of the plain definition (T = 6,
    # D = 1392, F = 192: Yb's worst ratio is 1.015, and so is the kernels';
    # with an fp32 H it would be 0.24).  So: the kernels must be within the
    # tolerance of Yb everywhere, and within that of Y wherever the prescribed
    # rounding alone stays below half of it.
    rows = np.arange(T) if T <= 64 else I.sample_rows(T, 40)
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=T * 31 + D + F)
    y = gmlp.forward(*(_dev(a) for a in (X, Wg, Wu, Wd)), workspace=gmlp.Workspace(T, D, F))
    torch.cuda.synchronize()
    got = I.bf16_bits_to_f32(gmlp.to_bf16_bits(y)[rows]).astype(np.float64)
    ref, h = orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows, return_h=True)
    ref_b = orc.down_rows(I.f32_to_bf16_bits(h.astype(np.float32)), Wd)
    bound = TOL * (np.abs(ref) + np.sqrt(np.mean(ref ** 2)))
    assert np.all(np.isfinite(got))
    r_b = np.abs(ref_b - ref) / bound        # the prescribed rounding alone
    r_gpu_b = np.abs(got - ref_b) / bound
    r_gpu = np.abs(got - ref) / bound
    waived = int(np.sum(r_b > 0.5))  # judged against Yb only (depends on the oracle alone)
    print("T=%d D=%d F=%d: max err/bound %.3f vs Y, %.3f vs Yb; rounding of H alone %.3f; "
          "%d of %d elements (%.3f%%) judged against Yb only"
          % (T, D, F, r_gpu.max(), r_gpu_b.max(), r_b.max(), waived, r_b.size, 100.0 * waived / r_b.size),
          flush=True)
    # At these seeds the rounding of H alone passes half the bound on at most
    # 0.23% of a shape's elements (0.04% over all sixteen shapes); the cap
    # keeps that exemption from growing unnoticed if the shapes change.
    assert waived <= WAIVER_CAP * r_b.size, (waived, r_b.size)
    assert np.all(r_gpu_b <= 1.0)
    assert np.all(r_gpu[r_b <= 0.5] <= 1.0)


@pytest.mark.parametrize("T", [1, 2, 5, 8])
def test_small_T_on_the_mfma_path(orc, T):
    _run(T, 264, 520, seed=40 + T, path="mfma", orc=orc)


# Up to 2 tokens the gate/up GEMV streams 512-column strips with one 1 KB row
# segment per wave and the down GEMV 256-column strips in 16 half-wave row
# groups: strips cut short by F or D, a single 8-column strip, splits shorter
# than one load batch (32 or 64 rows) and a last split cut short by K.
WIDE_GEMV = [(1, 8, 8), (1, 40, 1032), (2, 1032, 8), (2, 4104, 520), (1, 264, 14344), (2, 72, 24584)]


@pytest.mark.parametrize("T,D,F", WIDE_GEMV, ids=["T%dD%dF%d" % s for s in WIDE_GEMV])
def test_eight_wave_gemv_strips(orc, T, D, F):
    plan = gmlp.describe(T, D, F)
    assert plan[0][0].startswith("gemv") and plan[0][2] == 512 and plan[1][2] == 512
    _run(T, D, F, seed=3 * T + D + F, orc=orc)


# 65 to 192 tokens where the dual-B gate/up tiles would split K in two (or
# run two 128-token tiles) over more than 3/4 of the chip: a G and a U block
# per column tile, each over the whole of K, the later of the two combining
# both into H.  96-, 128- and 192-token tiles, K tails (D not a multiple of
# 64), last column tiles cut short by F (F = 12424, 14344, 12296), the
# fewest (97) and most (128) pairs.
PAIRED = [(65, 264, 12800), (96, 4104, 12424), (97, 264, 16384), (128, 1032, 14344), (112, 520, 12296),
          (129, 264, 14344), (160, 1032, 16384), (192, 520, 12424)]


@pytest.mark.parametrize("T,D,F", PAIRED, ids=["T%dD%dF%d" % s for s in PAIRED])
def test_paired_gate_up_blocks(orc, T, D, F):
    plan = gmlp.describe(T, D, F)
    assert plan[0][0].endswith(", 2, true, true>") and plan[0][3] == 2, plan
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=T + D + F)
    x, wg, wu, wd = (_dev(a) for a in (X, Wg, Wu, Wd))
    ws = gmlp.Workspace(T, D, F)
    rows = I.sample_rows(T, 24) if D * F > 2 ** 24 else np.arange(T)
    h = gmlp.gate_up(x, wg, wu, workspace=ws)
    y = gmlp.forward(x, wg, wu, wd, workspace=ws)
    torch.cuda.synchronize()
    Y_ref, H_ref = orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows, return_h=True)
    _check(gmlp.to_bf16_bits(h)[rows], H_ref, "paired H T=%d D=%d F=%d" % (T, D, F))
    _check(gmlp.to_bf16_bits(y)[rows], Y_ref, "paired Y T=%d D=%d F=%d" % (T, D, F))


@pytest.mark.parametrize("T,D,F", [(150, 8200, 4104), (137, 2056, 3080)])
def test_160_token_down_tiles(orc, T, D, F):
    # 129 to 160 tokens: one 160-token down tile split over K (ragged D and
    # F, 3 and 13 splits).
    assert gmlp.describe(T, D, F)[-1][0] == "gemm_mfma_kernel<GemmShape<1, 4, 1, 1, 5, 3, 64>, 1, true, true>"
    _run(T, D, F, seed=T + D, rows=np.unique(np.concatenate([I.sample_rows(T, 16), np.arange(T - 4, T)])), orc=orc)


# 257 to 384 tokens: two 192-token tiles in both steps (the gate/up step
# where they fill 3/4 of a round to one round, the down step where it has
# 64 to 128 tiles), with a ragged second token tile and ragged D and F.
TILES192 = [(257, 4040, 12296), (300, 4040, 14344), (384, 8136, 16384), (350, 3976, 12424), (320, 4040, 4104)]


@pytest.mark.parametrize("T,D,F", TILES192, ids=["T%dD%dF%d" % s for s in TILES192])
def test_192_token_tiles(orc, T, D, F):
    plan = gmlp.describe(T, D, F)
    assert "GemmShape<1, 4, 1, 1, 6, 3, 64>, 1, true, false>" in plan[-1][0], plan
    if F > 12160:
        assert plan[0][0] == "gemm_mfma_kernel<GemmShape<2, 4, 1, 1, 6, 4, 32>, 0, false, false>", plan
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=T + D + F)
    x, wg, wu, wd = (_dev(a) for a in (X, Wg, Wu, Wd))
    ws = gmlp.Workspace(T, D, F)
    rows = np.unique(np.concatenate([I.sample_rows(T, 16), np.arange(T - 8, T)])) if D * F > 2 ** 24 else np.arange(T)
    h = gmlp.gate_up(x, wg, wu, workspace=ws)
    y = gmlp.forward(x, wg, wu, wd, workspace=ws)
    torch.cuda.synchronize()
    Y_ref, H_ref = orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows, return_h=True)
    _check(gmlp.to_bf16_bits(h)[rows], H_ref, "192-token H T=%d D=%d F=%d" % (T, D, F))
    _check(gmlp.to_bf16_bits(y)[rows], Y_ref, "192-token Y T=%d D=%d F=%d" % (T, D, F))


# From 513 tokens the gate/up step may run on a token split: the whole
# 256-token tiles of the first T - r rows, then the last r rows as a
# problem of their own (GEMV kernels for r <= 5, few-token tiles, pairs).
TOKEN_SPLIT = [(515, 1032, 14344), (520, 264, 14344), (600, 1032, 14344), (1100, 520, 14344)]


@pytest.mark.parametrize("T,D,F", TOKEN_SPLIT, ids=["T%dD%dF%d" % s for s in TOKEN_SPLIT])
def test_gate_up_token_split(orc, T, D, F):
    r = T % 256
    plan = gmlp.describe(T, D, F)
    assert plan[0][0] == "gemm_mfma_kernel<GemmShape<2, 4, 2, 1, 4, 2, 64>, 0, false, false>", plan
    assert plan[1][0].startswith("gemv_splitk_kernel<%d, 2," % r) if r <= 5 else plan[1][3] == 2, plan
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=T + D + F)
    x, wg, wu, wd = (_dev(a) for a in (X, Wg, Wu, Wd))
    ws = gmlp.Workspace(T, D, F)
    edge = np.arange(T - r - 3, T - r + 3)
    rows = np.unique(np.concatenate([I.sample_rows(T, 16), edge, np.arange(T - 3, T)]))
    h = gmlp.gate_up(x, wg, wu, workspace=ws)
    y = gmlp.forward(x, wg, wu, wd, workspace=ws)
    torch.cuda.synchronize()
    Y_ref, H_ref = orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows, return_h=True)
    _check(gmlp.to_bf16_bits(h)[rows], H_ref, "token-split H T=%d D=%d F=%d" % (T, D, F))
    _check(gmlp.to_bf16_bits(y)[rows], Y_ref, "token-split Y T=%d D=%d F=%d" % (T, D, F))


# Each GEMV strip's arrival counter sits on a 128-byte line of its own
# where both steps' counters fit the counter block so (up to 512 strips in
# all); past that, on consecutive words.  514 strips (F = 262152): the
# consecutive words, for both the two-kernel and the one-kernel path.
@pytest.mark.parametrize("path", ["gemv", "fused"])
def test_gemv_with_more_strips_than_counter_lines(orc, path):
    T, D, F = 1, 264, 262152
    _run(T, D, F, seed=61, path=path, orc=orc)


@pytest.mark.parametrize("T", [1, 3, 8])
def test_gemv_path_explicitly(orc, T):
    _run(T, 4104, 2056, seed=50 + T, path="gemv", orc=orc)


def test_large_gate_up_tiles_ragged(orc):
    # 4 x 129 = 516 tiles of 256 x 128: the large gate/up configuration, with
    # ragged T, D (K tail of 8) and F (a partial 128-column tile).
    T, D, F = 1000, 264, 16392
    _run(T, D, F, seed=7, rows=I.sample_rows(T, 96), orc=orc)


def test_large_down_tiles_ragged(orc):
    # 16 x 13 = 208 tiles of 256 x 256: the large down configuration.
    T, D, F = 4000, 3080, 264
    _run(T, D, F, seed=8, rows=I.sample_rows(T, 64), orc=orc)


def test_gate_up_alone_matches_oracle_h(orc):
    for T, D, F in [(16, 256, 512), (5, 264, 1032), (200, 520, 264)]:
        X, Wg, Wu, Wd = I.generate(T, D, F, seed=3)
        h = gmlp.gate_up(_dev(X), _dev(Wg), _dev(Wu))
        torch.cuda.synchronize()
        _, H_ref = orc.gated_mlp_rows(X, Wg, Wu, Wd, return_h=True)
        _check(gmlp.to_bf16_bits(h), H_ref, "H T=%d D=%d F=%d" % (T, D, F))


def test_down_alone_matches_oracle(orc):
    for T, F, D in [(16, 512, 256), (3, 1032, 264), (130, 264, 520)]:
        rng = np.random.default_rng(T)
        H = I.f32_to_bf16_bits(rng.standard_normal((T, F)).astype(np.float32))
        Wd = I.f32_to_bf16_bits((rng.standard_normal((F, D)) / np.sqrt(F)).astype(np.float32))
        y = gmlp.down(_dev(H), _dev(Wd))
        torch.cuda.synchronize()
        _check(gmlp.to_bf16_bits(y), orc.down_rows(H, Wd), "down T=%d F=%d D=%d" % (T, F, D))


def test_forward_without_workspace_allocates_its_own(orc):
    X, Wg, Wu, Wd = I.generate(12, 256, 520, seed=9)
    y = gmlp.forward(_dev(X), _dev(Wg), _dev(Wu), _dev(Wd))
    torch.cuda.synchronize()
    _check(gmlp.to_bf16_bits(y), orc.gated_mlp_rows(X, Wg, Wu, Wd), "allocating entry")


def test_zero_tokens_leaves_output_untouched():
    X, Wg, Wu, Wd = I.generate(1, 256, 512, seed=0)
    y = torch.full((1, 256), 3.0, dtype=torch.bfloat16, device="cuda")
    x0 = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    y0 = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    gmlp.forward(x0, _dev(Wg), _dev(Wu), _dev(Wd), out=y0)
    torch.cuda.synchronize()
    assert torch.all(y == 3.0)


@pytest.mark.parametrize("T,D,F", [(1, 4096, 14336), (64, 1032, 2056), (100, 520, 12296), (600, 512, 4104)])
def test_bitwise_deterministic(T, D, F):
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=11)
    args = [_dev(a) for a in (X, Wg, Wu, Wd)]
    ws = gmlp.Workspace(T, D, F)
    a = gmlp.forward(*args, workspace=ws).clone()
    b = gmlp.forward(*args, workspace=ws).clone()
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("T", [3, 100, 1000])
def test_guard_bands_untouched(orc, T):
    """Writes stay inside Y: canary rows before and after it survive."""
    D, F = 264, 1032
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=12)
    pad = 7
    big = torch.full((T + 2 * pad, D), -77.0, dtype=torch.bfloat16, device="cuda")
    y = big[pad:pad + T]
    ws = gmlp.Workspace(T, D, F)
    gmlp.forward(*[_dev(a) for a in (X, Wg, Wu, Wd)], out=y, workspace=ws)
    torch.cuda.synchronize()
    assert torch.all(big[:pad] == -77.0) and torch.all(big[pad + T:] == -77.0)
    _check(gmlp.to_bf16_bits(y), orc.gated_mlp_rows(X, Wg, Wu, Wd), "guarded T=%d" % T)


def test_non_default_stream_and_ordering(orc):
    T, D, F = 40, 520, 1032
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=13)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        args = [_dev(a) for a in (X, Wg, Wu, Wd)]
        x = args[0] * 1.0  # work queued ahead of the call on the same stream
        y = gmlp.forward(x, *args[1:], stream=s)
        z = y.float() * 2.0  # work queued behind it
    s.synchronize()
    _check(gmlp.to_bf16_bits(y), orc.gated_mlp_rows(X, Wg, Wu, Wd), "side stream")
    assert torch.equal(z, y.float() * 2.0)


def test_workspace_reused_across_shapes(orc):
    ws = gmlp.Workspace(300, 1032, 2056)
    for T, D, F in [(300, 1032, 2056), (4, 1032, 2056), (100, 520, 1032), (1, 264, 264)]:
        assert ws.fits(T, D, F)
        X, Wg, Wu, Wd = I.generate(T, D, F, seed=T)
        y = gmlp.forward(*[_dev(a) for a in (X, Wg, Wu, Wd)], workspace=ws)
        torch.cuda.synchronize()
        _check(gmlp.to_bf16_bits(y), orc.gated_mlp_rows(X, Wg, Wu, Wd), "reuse T=%d" % T)


# ---- the five workloads at their full sizes ---------------------------------

@pytest.mark.parametrize("name,nrows", [("decode", None), ("small_batch", None),
                                        ("prefill", 64), ("large_prefill", 48)])
def test_full_size_workload(orc, name, nrows):
    w = I.WORKLOADS[name]
    rows = None if nrows is None else I.sample_rows(w.T, nrows)
    _run(w.T, w.D, w.F, seed=w.seed, rows=rows, unit_rms=w.unit_rms_rows, orc=orc)


@pytest.mark.parametrize("T", [16, 48, 80])
def test_few_token_tiles_at_model_dims(orc, T):
    # The 32-, 64- and 96-token tile configurations at the decode model's D
    # and F (split-K over D = 4096 and F = 14336), on sampled rows.
    _run(T, 4096, 14336, seed=60 + T, rows=I.sample_rows(T, 8), orc=orc)


@pytest.mark.parametrize("T,D,F", [(704, 264, 14336), (4096, 4352, 2056)])
def test_tail_tiles_split_over_k(orc, T, D, F):
    # 256-token tiles that leave a last round of blocks at most half full:
    # the whole rounds run as one launch, the remaining tiles as a second,
    # split-K launch (T = 704: 336 gate/up tiles = 256 + 80 split 2 ways;
    # the second shape has tails in both steps, 272 tiles each).
    plan = gmlp.describe(T, D, F)
    assert any(", true, false>" in k and "GemmShape<2, 4, 2, 1, 4" in k for k, *_ in plan)
    _run(T, D, F, seed=T + F, rows=I.sample_rows(T, 48), orc=orc)
    # Fixed-order reductions: a second call gives the same bits.
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=T + F)
    args = [_dev(a) for a in (X, Wg, Wu, Wd)]
    a = gmlp.forward(*args).clone()
    b = gmlp.forward(*args)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("T,D,F", [(448, 4104, 14336), (600, 2056, 14344), (1280, 2056, 13000)])
def test_wide_down_tiles_split_over_k(orc, T, D, F):
    # Above 256 tokens, where few down tiles fill the chip only with short
    # splits, 256 x 128 down tiles split over K (ragged T, D and F in the
    # second shape); fixed-order reduction: a second call gives the same bits.
    plan = gmlp.describe(T, D, F)
    assert plan[-1][0] == "gemm_mfma_kernel<GemmShape<1, 4, 2, 2, 2, 3, 64>, 1, true, false>" and plan[-1][3] > 1
    _run(T, D, F, seed=T + D, rows=I.sample_rows(T, 24), orc=orc)
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=T + D)
    args = [_dev(a) for a in (X, Wg, Wu, Wd)]
    a = gmlp.forward(*args).clone()
    b = gmlp.forward(*args)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("T,D,F", [(257, 264, 24584), (300, 136, 24584), (513, 264, 12296)])
def test_large_gate_up_tiles_above_256_tokens(orc, T, D, F):
    # Above 256 tokens the 256-token gate/up tiles are used once they nearly
    # fill the chip; ragged token tails and column tails on that path.
    assert gmlp.describe(T, D, F)[0][0].startswith("gemm_mfma_kernel<GemmShape<2, 4, 2, 1, 4,")
    _run(T, D, F, seed=T + F, orc=orc)


@pytest.mark.parametrize("T,D,F", [(1, 4096, 14336), (48, 4096, 14336), (600, 1032, 2056)])
def test_h_is_rounded_once_to_nearest_even(orc, T, D, F):
    """H is the fp32 value act(G) * U rounded once to bf16, to nearest even.
    The kernel's fp32 H differs from the oracle's fp64 H by a few parts in a
    million, so it rounds to the same bf16 as the fp64 value except near a
    rounding boundary (expected: well under 1% of elements), and never more
    than one bf16 step away.  The tolerance of the Y tests cannot see the
    rounding mode (H truncated instead stays within it); truncation or a
    second rounding would leave about half the elements one step off here."""
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=500 + T)
    h = gmlp.gate_up(_dev(X), _dev(Wg), _dev(Wu), workspace=gmlp.Workspace(T, D, F))
    torch.cuda.synchronize()
    got = gmlp.to_bf16_bits(h).astype(np.int32)
    rows = np.arange(T) if T <= 64 else I.sample_rows(T, 64)
    _, H_ref = orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows, return_h=True)
    want = I.f32_to_bf16_bits(H_ref.astype(np.float32)).astype(np.int32)
    got = got[rows]
    same = float(np.mean(got == want))
    # Adjacent bf16 values of one sign have adjacent bit patterns.  Within a
    # few fp32 accumulation errors of zero the sign itself is not determined,
    # so the one-step check leaves out |H| below 1e-3 of its rms.
    away = np.abs(H_ref) >= 1e-3 * np.sqrt(np.mean(H_ref ** 2))
    steps = np.abs(got - want)[away]
    print("T=%d D=%d F=%d: %.4f%% of H equal to the fp64 H rounded to nearest even, max %d step(s)"
          % (T, D, F, 100 * same, int(steps.max())), flush=True)
    assert same >= 0.99
    assert steps.max() <= 1


@pytest.mark.parametrize("T,D,F,splits", [(1280, 4104, 13000, 3), (2304, 4104, 264, 1)])
def test_large_down_tiles_below_a_round(orc, T, D, F, splits):
    # 40 to 191 tiles of 256 x 256 for the down step: split over K to fill a
    # round (3 splits of 68 k-tiles for 85 tiles, where 256 x 128 tiles
    # would take more than a round), or, with 129 tiles or more, one partial
    # round without split-K.
    (name, grid, block, k_splits) = gmlp.describe(T, D, F)[-1]
    assert name.startswith("gemm_mfma_kernel<GemmShape<1, 4, 2, 2, 4, 2, 64>") and k_splits == splits
    _run(T, D, F, seed=T + D, rows=I.sample_rows(T, 48), orc=orc)
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=T + D)
    args = [_dev(a) for a in (X, Wg, Wu, Wd)]
    ws = gmlp.Workspace(T, D, F)
    a = gmlp.forward(*args, workspace=ws).clone()
    b = gmlp.forward(*args, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
