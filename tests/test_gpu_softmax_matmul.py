"""GPU parity for Softmax+MatMul: the HIP path (through the C ABI) against the
CPU fp64 oracle of Fig. fig:softmax-matmul-comp-graph (a).

Acceptance per output element: |Z_gpu - Z_ref| <= 1e-2 * (|Z_ref| + rms(Z_ref)),
rms over the checked elements (bf16 inputs, P = exp(X - rowmax) rounded to
bf16, fp32 accumulation and division, Z rounded to bf16).  Small shapes are
checked in full; the 8192^3 benchmark shape on sampled rows, in the launch
configuration the benchmark times.  Cases outside the oracle's domain (logits
beyond double's exp range) are checked through properties that hold at any
size: shift invariance and a dominant logit selecting a row of Y.
"""
import numpy as np
import pytest
import torch

from paper_2606_26344_amd import gmlp
from paper_2606_26344_amd import inputs as I
from paper_2606_26344_amd import softmax_matmul as smm

pytestmark = pytest.mark.gpu

TOL = 1e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    gmlp.library()  # fails loudly when libgmlp.so is missing


@pytest.fixture(scope="module")
def sorc():
    import oracle

    return oracle.softmax_matmul.default_oracle()


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


def _gpu_run(X, Y, path="auto", workspace=None):
    z = smm.softmax_matmul(_dev(X), _dev(Y), path=path, workspace=workspace)
    torch.cuda.synchronize()
    return gmlp.to_bf16_bits(z)


def _run(sorc, M, K, N, seed=0, path="auto", scale=1.0, rows=None):
    X, Y = I.generate_softmax_matmul(M, K, N, seed=seed, logit_scale=scale)
    print("softmax_matmul M=%d K=%d N=%d path=%s scale=%g seed=%d" % (M, K, N, path, scale, seed),
          flush=True)
    Z = _gpu_run(X, Y, path=path)
    if rows is None:
        rows = np.arange(M)
    ref = sorc.rows(X, Y, rows=rows)
    return _check(Z[rows], ref, "M=%d K=%d N=%d path=%s scale=%g" % (M, K, N, path, scale))


def test_tiny_workload(sorc):
    w = I.SOFTMAX_MATMUL_WORKLOADS["softmax_matmul_tiny"]
    _run(sorc, w.M, w.K, w.N, seed=w.seed)


# Ragged shapes (K, N multiples of 8 only), every row-kernel width (K up to
# 512 columns per chunk-per-lane step: 1, 2, 4, 8, 16 chunks, and K > 8192
# streamed in two passes), both matmul paths and both MFMA tile sizes.
SHAPES = [
    (1, 8, 8), (1, 264, 520), (2, 1000, 264), (3, 520, 1032), (5, 2056, 72), (8, 4104, 264),
    (9, 136, 264), (16, 256, 512), (33, 1032, 136), (64, 8192, 264), (127, 520, 1032),
    (129, 264, 520), (300, 2056, 1032), (24, 9000, 136), (4, 16392, 64),
]


@pytest.mark.parametrize("M,K,N", SHAPES, ids=["M%dK%dN%d" % s for s in SHAPES])
def test_shapes(sorc, M, K, N):
    _run(sorc, M, K, N, seed=M + K + N)


@pytest.mark.parametrize("M", [1, 3, 8])
def test_small_M_on_the_mfma_path(sorc, M):
    _run(sorc, M, 1032, 520, seed=7 + M, path="mfma")


@pytest.mark.parametrize("scale", [0.0, 4.0, 16.0])
def test_logit_scales(sorc, scale):
    # scale 0: every logit 0, softmax uniform, Z = column means of Y;
    # larger scales: peaked rows dominated by a few logits.
    _run(sorc, 40, 2056, 264, seed=11, scale=scale)


def test_benchmark_shape_sampled_rows(sorc):
    w = I.SOFTMAX_MATMUL_WORKLOADS["softmax_matmul"]
    rows = I.sample_rows(w.M, n=48)
    _run(sorc, w.M, w.K, w.N, seed=w.seed, rows=rows)


def test_matmul_tail_tiles_split_over_k(sorc):
    # 16 x 17 = 272 tiles of 256 x 256: one round of whole tiles, then, in
    # the same launch, 16 tiles split over K.
    M, K, N = 4096, 2056, 4352
    plan = smm.describe(M, K, N)
    assert len(plan) == 2 and plan[1][3] > 1 and plan[1][1] == 256 + 16 * plan[1][3], plan
    _run(sorc, M, K, N, seed=41, rows=I.sample_rows(M, 32))


def test_matmul_on_wide_tiles_split_over_k(sorc):
    # 2 x 17 = 34 tiles of 256 x 128 (a ragged second row tile), 3 splits:
    # the divide by the softmax sums in the split-K epilogue of the wide
    # tiles.
    M, K, N = 448, 16384, 4104
    assert smm.describe(M, K, N)[-1][0] == "gemm_mfma_kernel<GemmShape<1, 4, 2, 2, 2, 3, 64>, 1, true, false>"
    _run(sorc, M, K, N, seed=43, rows=I.sample_rows(M, 24))


def test_matmul_on_192_row_tiles_split_over_k(sorc):
    # 257 to 384 rows: two 192-row tiles split over K, the second ragged.
    M, K, N = 300, 16384, 4040
    assert smm.describe(M, K, N)[-1][0] == "gemm_mfma_kernel<GemmShape<1, 4, 1, 1, 6, 3, 64>, 1, true, false>"
    _run(sorc, M, K, N, seed=44, rows=I.sample_rows(M, 24))


def test_probabilities_past_2_gib(sorc):
    """X and P = exp(X - rowmax) of more than 2 GiB each (M = 131080,
    K = 8192): row and tile base addresses are formed in 64 bits.  The
    checked rows include the last ones, which lie past 2 GiB."""
    M, K, N = 131080, 8192, 264
    assert M * K * 2 > 2 ** 31
    rows = np.array([0, 1, 65536, 131071, 131072, 131079])
    _run(sorc, M, K, N, seed=43, rows=rows)


def test_gemv_and_mfma_paths_agree(sorc):
    X, Y = I.generate_softmax_matmul(6, 4096, 1032, seed=3)
    ref = sorc.rows(X, Y)
    for path in ("gemv", "mfma"):
        _check(_gpu_run(X, Y, path=path), ref, "M=6 path=%s" % path)


def test_deterministic_and_workspace_reuse():
    # The same call twice, and a smaller call in between on the same
    # workspace: bit-identical results (fixed-order reductions).
    X, Y = I.generate_softmax_matmul(100, 4096, 520, seed=5)
    X2, Y2 = I.generate_softmax_matmul(3, 1024, 520, seed=6)
    ws = smm.make_workspace(100, 4096, 520)
    a = _gpu_run(X, Y, workspace=ws)
    _gpu_run(X2, Y2, workspace=ws)
    b = _gpu_run(X, Y, workspace=ws)
    assert np.array_equal(a, b)


def test_shift_invariance_beyond_the_oracle_domain():
    # Logits near 1000 overflow exp in double precision, so the oracle cannot
    # evaluate them; softmax is unchanged by a per-row shift.  Logits that are
    # multiples of 4 in [-20, 20] shifted by 1000 stay exact in bf16 and
    # x - rowmax is exact in fp32, so the results must be bit-identical.
    r = np.random.default_rng(21)
    X0f = 4.0 * r.integers(-5, 6, size=(12, 1032)).astype(np.float32)
    X0 = I.f32_to_bf16_bits(X0f)
    Xc = I.f32_to_bf16_bits(X0f + 1000.0)
    assert np.array_equal(I.bf16_bits_to_f32(Xc) - 1000.0, X0f)
    _, Y = I.generate_softmax_matmul(1, 1032, 264, seed=22)
    for path in ("gemv", "mfma"):
        assert np.array_equal(_gpu_run(X0[:8], Y, path=path), _gpu_run(Xc[:8], Y, path=path))
    assert np.array_equal(_gpu_run(X0, Y), _gpu_run(Xc, Y))


def test_dominant_logit_selects_a_row_of_y():
    # One logit 200 above the rest of its row: every other exponential
    # underflows in fp32, s = 1 exactly, and Z is that row of Y, bit for bit.
    M, K, N = 20, 2056, 264
    hot = np.random.default_rng(23).integers(0, K, size=M)
    Xf = np.zeros((M, K), np.float32)
    Xf[np.arange(M), hot] = 200.0
    _, Y = I.generate_softmax_matmul(1, K, N, seed=24)
    X = I.f32_to_bf16_bits(Xf)
    assert np.array_equal(_gpu_run(X, Y, path="mfma"), Y[hot])
    assert np.array_equal(_gpu_run(X[:8], Y, path="gemv"), Y[hot[:8]])


def test_nan_row_gives_nan_row():
    X, Y = I.generate_softmax_matmul(10, 520, 136, seed=25)
    X[3, 77] = 0x7FC0  # a quiet NaN
    Z = I.bf16_bits_to_f32(_gpu_run(X, Y))
    assert np.all(np.isnan(Z[3]))
    assert np.all(np.isfinite(np.delete(Z, 3, axis=0)))


def test_zero_rows_is_a_no_op():
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((64, 16), dtype=torch.bfloat16, device="cuda")
    z = smm.softmax_matmul(x, y)
    torch.cuda.synchronize()
    assert z.shape == (0, 16)


def test_halves_compose_to_the_whole_call(sorc):
    # exp_rows then divide gives softmax_matmul's bits; P / s is the softmax
    # the oracle computes, within the bf16 rounding of P (at most 2^-8
    # relative) plus the fp32 error of exp and of the sum s (below 1e-3).
    for M, K, N in [(6, 4096, 520), (70, 1032, 264)]:
        X, Y = I.generate_softmax_matmul(M, K, N, seed=31 + M, logit_scale=3.0)
        x, y = _dev(X), _dev(Y)
        p, s = smm.exp_rows(x)
        z = smm.divide(p, s, y)
        torch.cuda.synchronize()
        assert np.array_equal(gmlp.to_bf16_bits(z), _gpu_run(X, Y))
        _, A = sorc.rows(X, Y, return_softmax=True)
        P = I.bf16_bits_to_f32(gmlp.to_bf16_bits(p)).astype(np.float64)
        S = s.cpu().numpy().astype(np.float64)
        assert np.all(S >= 1.0) and np.all(S <= K)
        err = np.abs(P / S[:, None] - A)
        assert np.all(err <= (2.0 ** -8 + 1e-3) * A + 1e-30), float(np.max(err / (A + 1e-30)))
