"""GPU checks of the fused decode kernel (GMLP_PATH_FUSED): the whole Gated
MLP for T <= 8 in one launch, the gate/up items on the first blocks and the
down items on the rest, each down block waiting only for the strips of H
its rows read.

It runs the same items and reductions as the two-kernel GEMV path, so its Y
must equal that path's bit for bit; it is also held to the oracle's
tolerance |Y - Y_ref| <= 1e-2 (|Y_ref| + rms(Y_ref)).
"""
import numpy as np
import pytest
import torch

from paper_2606_26344_amd import gmlp
from paper_2606_26344_amd import inputs as I

pytestmark = pytest.mark.gpu

TOL = 1e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    gmlp.library()


def _run(X, Wg, Wu, Wd, path, ws=None, **variant):
    y = gmlp.forward(*(gmlp.from_bf16_bits(a) for a in (X, Wg, Wu, Wd)), path=path, workspace=ws,
                     **variant)
    torch.cuda.synchronize()
    return gmlp.to_bf16_bits(y)


def _check(got_bits, ref, what):
    got = I.bf16_bits_to_f32(got_bits).astype(np.float64)
    rms = float(np.sqrt(np.mean(ref ** 2)))
    err = np.abs(got - ref)
    bound = TOL * (np.abs(ref) + rms)
    ratio = float(np.max(err / bound))
    print("%s max err/bound = %.3f" % (what, ratio), flush=True)
    assert np.all(err <= bound), what


SHAPES = [(T, 264, 520) for T in range(1, 9)] + [(1, 72, 136), (5, 1032, 72), (8, 2056, 1032)]


@pytest.mark.parametrize("T,D,F", SHAPES, ids=["T%dD%dF%d" % s for s in SHAPES])
def test_fused_equals_two_kernels_and_oracle(orc, T, D, F):
    print("fused T=%d D=%d F=%d" % (T, D, F), flush=True)
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=100 + T + D)
    fused = _run(X, Wg, Wu, Wd, "fused")
    assert np.array_equal(fused, _run(X, Wg, Wu, Wd, "gemv"))
    _check(fused, orc.gated_mlp_rows(X, Wg, Wu, Wd), "fused T=%d D=%d F=%d" % (T, D, F))


@pytest.mark.parametrize("T", [1, 2, 8])
def test_fused_decode_shape(orc, T):
    print("fused decode T=%d" % T, flush=True)
    X, Wg, Wu, Wd = I.generate(T, 4096, 14336, seed=T)
    fused = _run(X, Wg, Wu, Wd, "fused")
    assert np.array_equal(fused, _run(X, Wg, Wu, Wd, "gemv"))
    _check(fused, orc.gated_mlp_rows(X, Wg, Wu, Wd), "fused decode T=%d" % T)


@pytest.mark.parametrize("variant", [dict(rmsnorm=True, eps=1e-5),
                                     dict(activation="swish", beta=1.702, rmsnorm=True, eps=1e-6),
                                     dict(activation="sigmoid")],
                         ids=["rmsnorm", "rmsnorm_swiglu", "glu"])
def test_fused_variants(orc, variant):
    X, Wg, Wu, Wd = I.generate(3, 1032, 2056, seed=7)
    fused = _run(X, Wg, Wu, Wd, "fused", **variant)
    assert np.array_equal(fused, _run(X, Wg, Wu, Wd, "gemv", **variant))
    _check(fused, orc.gated_mlp_rows(X, Wg, Wu, Wd, **variant), "fused %s" % variant)


def test_fused_repeated_calls_on_one_workspace():
    # The barrier's count and flags return to zero: back-to-back calls, and a
    # call of another shape in between, give the same bits.
    X, Wg, Wu, Wd = I.generate(4, 1032, 2056, seed=9)
    X2, Wg2, Wu2, Wd2 = I.generate(2, 264, 520, seed=10)
    ws = gmlp.Workspace(4, 1032, 2056)
    first = _run(X, Wg, Wu, Wd, "fused", ws)
    for _ in range(3):
        _run(X2, Wg2, Wu2, Wd2, "fused", ws)
        assert np.array_equal(_run(X, Wg, Wu, Wd, "fused", ws), first)


def test_fused_next_to_a_kernel_on_another_stream():
    # The waits of the fused kernel are on blocks of lower index only, which
    # the hardware dispatches first, so the kernel completes with the same
    # bits while another stream's kernel holds part of the chip (here a
    # prefill-sized GEMM step running concurrently, both streams at the
    # default priority).
    X, Wg, Wu, Wd = I.generate(3, 4096, 14336, seed=12)
    ref = _run(X, Wg, Wu, Wd, "gemv")
    Xb, Wgb, Wub, Wdb = I.generate(2048, 1024, 4096, seed=13)
    big = [gmlp.from_bf16_bits(a) for a in (Xb, Wgb, Wub, Wdb)]
    ws_big = gmlp.Workspace(2048, 1024, 4096)
    args = [gmlp.from_bf16_bits(a) for a in (X, Wg, Wu, Wd)]
    ws = gmlp.Workspace(3, 4096, 14336)
    y = torch.empty((3, 4096), dtype=torch.bfloat16, device="cuda")
    other, mine = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for _ in range(5):
        with torch.cuda.stream(other):
            for _ in range(4):
                gmlp.forward(*big, workspace=ws_big)
        with torch.cuda.stream(mine):
            gmlp.forward(*args, out=y, path="fused", workspace=ws)
        torch.cuda.synchronize()
        assert np.array_equal(gmlp.to_bf16_bits(y), ref)


# Counter block at the start of a workspace: GEMV strip and GEMM tile
# counters (64 KiB), the fused kernel's ready words (64 KiB), then the line
# with its give-up count.
COUNTER_BLOCK_BYTES = 64 * 1024 + 64 * 1024 + 256


def test_fused_wait_that_gives_up_poisons_y_and_recovers():
    # A zero poll limit, set from the host, makes every down block whose
    # strips of H are not written yet give up at once; every kernel still runs
    # to completion.  At the decode shape the down blocks start alongside the
    # gate/up blocks, which take tens of microseconds, so some give up.
    T, D, F = 1, 4096, 14336
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=21)
    ref = _run(X, Wg, Wu, Wd, "gemv")
    ws = gmlp.Workspace(T, D, F)
    assert ws.fused_giveups() == 0
    prev = gmlp.fused_spin_limit(0)
    try:
        bad = _run(X, Wg, Wu, Wd, "fused", ws)
    finally:
        gmlp.fused_spin_limit(prev)
    giveups = ws.fused_giveups()
    nan = np.isnan(I.bf16_bits_to_f32(bad))
    print("fused give-ups: %d blocks, %d of %d outputs NaN" % (giveups, nan.sum(), nan.size), flush=True)
    assert giveups > 0 and nan.any()
    # A block that gave up turns the whole 256-column strip of Y it feeds to
    # NaN; every other strip has the two-kernel path's bits.
    for c0 in range(0, D, 256):
        strip = slice(c0, c0 + 256)
        assert nan[:, strip].all() or np.array_equal(bad[:, strip], ref[:, strip]), c0
    # Counters and ready words are back at zero; reading the give-up count
    # cleared it.
    assert int(torch.count_nonzero(ws.buffer[:COUNTER_BLOCK_BYTES])) == 0
    # The next call on the same workspace is bit-exact and gives up nowhere.
    for _ in range(2):
        assert np.array_equal(_run(X, Wg, Wu, Wd, "fused", ws), ref)
    assert ws.fused_giveups() == 0


def test_fused_ready_words_return_to_zero():
    X, Wg, Wu, Wd = I.generate(8, 2056, 1032, seed=22)
    ws = gmlp.Workspace(8, 2056, 1032)
    _run(X, Wg, Wu, Wd, "fused", ws)
    assert int(torch.count_nonzero(ws.buffer[:COUNTER_BLOCK_BYTES])) == 0
    assert ws.fused_giveups() == 0


# ---- the one-launch MFMA path (GMLP_PATH_FUSED_MFMA, T <= 64) ----------------

MFMA_SHAPES = [(1, 264, 520), (7, 256, 1032), (16, 520, 1032), (31, 264, 264), (32, 1032, 2056),
               (33, 264, 520), (48, 4104, 2056), (64, 520, 264), (5, 72, 136), (20, 2056, 72)]


@pytest.mark.parametrize("T,D,F", MFMA_SHAPES, ids=["T%dD%dF%d" % s for s in MFMA_SHAPES])
def test_fused_mfma_equals_two_kernels_and_oracle(orc, T, D, F):
    print("fused_mfma T=%d D=%d F=%d" % (T, D, F), flush=True)
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=200 + T + D)
    fused = _run(X, Wg, Wu, Wd, "fused_mfma")
    assert np.array_equal(fused, _run(X, Wg, Wu, Wd, "mfma"))
    _check(fused, orc.gated_mlp_rows(X, Wg, Wu, Wd), "fused_mfma T=%d D=%d F=%d" % (T, D, F))


@pytest.mark.parametrize("T", [8, 32, 64])
def test_fused_mfma_decode_model_dims(orc, T):
    print("fused_mfma model dims T=%d" % T, flush=True)
    X, Wg, Wu, Wd = I.generate(T, 4096, 14336, seed=T + 70)
    fused = _run(X, Wg, Wu, Wd, "fused_mfma")
    assert np.array_equal(fused, _run(X, Wg, Wu, Wd, "mfma"))
    rows = I.sample_rows(T, 8)
    _check(fused[rows], orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows), "fused_mfma decode dims T=%d" % T)


@pytest.mark.parametrize("variant", [dict(rmsnorm=True, eps=1e-5),
                                     dict(activation="swish", beta=1.702, rmsnorm=True, eps=1e-6),
                                     dict(activation="sigmoid")],
                         ids=["rmsnorm", "rmsnorm_swiglu", "glu"])
def test_fused_mfma_variants(orc, variant):
    X, Wg, Wu, Wd = I.generate(40, 1032, 2056, seed=8)
    fused = _run(X, Wg, Wu, Wd, "fused_mfma", **variant)
    assert np.array_equal(fused, _run(X, Wg, Wu, Wd, "mfma", **variant))
    _check(fused, orc.gated_mlp_rows(X, Wg, Wu, Wd, **variant), "fused_mfma %s" % variant)


def test_fused_mfma_repeated_calls_and_counters_return_to_zero():
    X, Wg, Wu, Wd = I.generate(24, 1032, 2056, seed=23)
    X2, Wg2, Wu2, Wd2 = I.generate(60, 264, 520, seed=24)
    ws = gmlp.Workspace(60, 1032, 2056)
    assert ws.fits(24, 1032, 2056) and ws.fits(60, 264, 520)
    first = _run(X, Wg, Wu, Wd, "fused_mfma", ws)
    for _ in range(3):
        _run(X2, Wg2, Wu2, Wd2, "fused_mfma", ws)
        assert np.array_equal(_run(X, Wg, Wu, Wd, "fused_mfma", ws), first)
    assert int(torch.count_nonzero(ws.buffer[:COUNTER_BLOCK_BYTES])) == 0
    assert ws.fused_giveups() == 0


def test_fused_mfma_wait_that_gives_up_poisons_y_and_recovers():
    # As for the decode kernel: a zero poll limit makes down blocks whose
    # rows of H are not written yet give up at once; every kernel completes.
    T, D, F = 16, 4096, 14336
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=25)
    ref = _run(X, Wg, Wu, Wd, "mfma")
    ws = gmlp.Workspace(T, D, F)
    prev = gmlp.fused_spin_limit(0)
    try:
        bad = _run(X, Wg, Wu, Wd, "fused_mfma", ws)
    finally:
        gmlp.fused_spin_limit(prev)
    giveups = ws.fused_giveups()
    nan = np.isnan(I.bf16_bits_to_f32(bad))
    print("fused_mfma give-ups: %d blocks, %d of %d outputs NaN" % (giveups, nan.sum(), nan.size), flush=True)
    assert giveups > 0 and nan.any()
    # A down block that gave up makes its whole 128-column tile of Y NaN;
    # every other tile has the two-kernel path's bits.
    for c0 in range(0, D, 128):
        tile = slice(c0, c0 + 128)
        assert nan[:, tile].all() or np.array_equal(bad[:, tile], ref[:, tile]), c0
    assert int(torch.count_nonzero(ws.buffer[:COUNTER_BLOCK_BYTES])) == 0
    for _ in range(2):
        assert np.array_equal(_run(X, Wg, Wu, Wd, "fused_mfma", ws), ref)
    assert ws.fused_giveups() == 0


def test_fused_mfma_next_to_a_kernel_on_another_stream():
    X, Wg, Wu, Wd = I.generate(20, 4096, 14336, seed=26)
    ref = _run(X, Wg, Wu, Wd, "mfma")
    Xb, Wgb, Wub, Wdb = I.generate(2048, 1024, 4096, seed=13)
    big = [gmlp.from_bf16_bits(a) for a in (Xb, Wgb, Wub, Wdb)]
    ws_big = gmlp.Workspace(2048, 1024, 4096)
    args = [gmlp.from_bf16_bits(a) for a in (X, Wg, Wu, Wd)]
    ws = gmlp.Workspace(20, 4096, 14336)
    y = torch.empty((20, 4096), dtype=torch.bfloat16, device="cuda")
    other, mine = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for _ in range(5):
        with torch.cuda.stream(other):
            for _ in range(4):
                gmlp.forward(*big, workspace=ws_big)
        with torch.cuda.stream(mine):
            gmlp.forward(*args, out=y, path="fused_mfma", workspace=ws)
        torch.cuda.synchronize()
        assert np.array_equal(gmlp.to_bf16_bits(y), ref)
    assert ws.fused_giveups() == 0
