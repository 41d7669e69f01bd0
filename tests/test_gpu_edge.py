"""Degenerate inputs of the Gated MLP on every kernel path.

* Structural zeros: Wg = 0 gives G = 0 and silu(0) = 0, Wu = 0 gives U = 0,
  X = 0 gives G = U = 0; each makes H = 0 and so Y = 0 exactly (no rounding
  can produce anything else).
* One-hot rows of X select rows of Wg and Wu, checked against the oracle.
* Rows are independent: a NaN in one row of X makes that row of Y NaN and
  leaves every other row finite and equal to the result without it.
"""
import numpy as np
import pytest
import torch

from paper_2606_26344_amd import gmlp
from paper_2606_26344_amd import inputs as I

pytestmark = pytest.mark.gpu

PATHS = [(3, "gemv"), (2, "fused"), (5, "mfma"), (64, "auto"), (80, "auto"), (128, "auto"), (300, "auto")]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    gmlp.library()


def _run(X, Wg, Wu, Wd, path, **variant):
    y = gmlp.forward(*(gmlp.from_bf16_bits(a) for a in (X, Wg, Wu, Wd)), path=path, **variant)
    torch.cuda.synchronize()
    return gmlp.to_bf16_bits(y)


@pytest.mark.parametrize("T,path", PATHS, ids=["T%d-%s" % p for p in PATHS])
@pytest.mark.parametrize("zero", ["Wg", "Wu", "X"])
def test_structural_zeros_give_exact_zero(T, path, zero):
    print("zeros %s T=%d path=%s" % (zero, T, path), flush=True)
    X, Wg, Wu, Wd = I.generate(T, 264, 520, seed=T)
    arrays = {"X": X, "Wg": Wg, "Wu": Wu}
    arrays[zero] = np.zeros_like(arrays[zero])
    Y = I.bf16_bits_to_f32(_run(arrays["X"], arrays["Wg"], arrays["Wu"], Wd, path))
    assert np.all(Y == 0.0)


@pytest.mark.parametrize("T,path", PATHS, ids=["T%d-%s" % p for p in PATHS])
def test_one_hot_rows(orc, T, path):
    D, F = 264, 520
    _, Wg, Wu, Wd = I.generate(1, D, F, seed=11)
    hot = np.random.default_rng(T).integers(0, D, size=T)
    Xf = np.zeros((T, D), np.float32)
    Xf[np.arange(T), hot] = 1.0
    X = I.f32_to_bf16_bits(Xf)
    got = I.bf16_bits_to_f32(_run(X, Wg, Wu, Wd, path)).astype(np.float64)
    ref = orc.gated_mlp_rows(X, Wg, Wu, Wd)
    bound = 1e-2 * (np.abs(ref) + np.sqrt(np.mean(ref ** 2)))
    assert np.all(np.abs(got - ref) <= bound)


@pytest.mark.parametrize("T,path", PATHS, ids=["T%d-%s" % p for p in PATHS])
@pytest.mark.parametrize("rmsnorm", [False, True])
def test_nan_row_stays_in_its_row(T, path, rmsnorm):
    X, Wg, Wu, Wd = I.generate(T, 264, 520, seed=5 + T)
    clean = _run(X, Wg, Wu, Wd, path, rmsnorm=rmsnorm)
    bad = T // 2
    Xn = X.copy()
    Xn[bad, 17] = 0x7FC0  # a quiet NaN
    Y = _run(Xn, Wg, Wu, Wd, path, rmsnorm=rmsnorm)
    assert np.all(np.isnan(I.bf16_bits_to_f32(Y[bad])))
    others = np.arange(T) != bad
    assert np.array_equal(Y[others], clean[others])


def test_concurrent_calls_on_two_streams_with_their_own_workspaces():
    # The library keeps no device state of its own: split-K counters and
    # partial sums live in the caller's workspace, so two streams running
    # calls at the same time, each with its workspace, give the bits of
    # sequential calls (split-K GEMM at T = 128 and 16, GEMV at T = 3).
    cases = [I.generate(T, 1032, 2056, seed=70 + T) for T in (128, 16, 3)]
    dev = [[gmlp.from_bf16_bits(a) for a in c] for c in cases]
    ref = []
    for args in dev:
        ref.append(gmlp.to_bf16_bits(gmlp.forward(*args, workspace=gmlp.Workspace(args[0].shape[0], 1032, 2056))))
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    wss = [[gmlp.Workspace(a[0].shape[0], 1032, 2056) for a in dev] for _ in streams]
    outs = [[torch.empty((a[0].shape[0], 1032), dtype=torch.bfloat16, device="cuda") for a in dev]
            for _ in streams]
    torch.cuda.synchronize()
    for _ in range(3):
        for s, st in enumerate(streams):
            with torch.cuda.stream(st):
                for rep in range(4):
                    for i, args in enumerate(dev):
                        gmlp.forward(*args, out=outs[s][i], workspace=wss[s][i])
        torch.cuda.synchronize()
        for s in range(len(streams)):
            for i in range(len(dev)):
                assert np.array_equal(gmlp.to_bf16_bits(outs[s][i]), ref[i])


@pytest.mark.parametrize("path", ["mfma", "gemv"])
def test_temporary_workspace_on_a_side_stream(orc, path):
    # forward() on a stream other than the current one, without a workspace:
    # the binding allocates the temporary workspace (and the output) on that
    # stream, so allocations made on the current stream right after the call
    # cannot be handed its memory while the kernels still use it.
    T, D, F = 6, 1032, 2056
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=31)
    args = [gmlp.from_bf16_bits(a) for a in (X, Wg, Wu, Wd)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    outs = []
    for _ in range(4):
        outs.append(gmlp.forward(*args, path=path, stream=s))
        junk = torch.full((1 << 22,), 7, dtype=torch.int32, device="cuda")  # current stream
        del junk
    s.synchronize()
    torch.cuda.synchronize()
    ref = orc.gated_mlp_rows(X, Wg, Wu, Wd)
    first = gmlp.to_bf16_bits(outs[0])
    for y in outs:
        assert np.array_equal(gmlp.to_bf16_bits(y), first)
    got = I.bf16_bits_to_f32(first).astype(np.float64)
    assert np.all(np.abs(got - ref) <= 1e-2 * (np.abs(ref) + np.sqrt(np.mean(ref ** 2))))
