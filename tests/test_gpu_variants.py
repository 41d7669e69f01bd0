"""GPU parity of the Gated MLP family against the CPU fp64 oracle.

Members: the gate activation swish_beta(g) = g * sigmoid(beta g) (SwiGLU) or
sigmoid(g) (GLU) in place of silu, and RMSNorm of X in front (the equation
of Section 2, applied by the kernels after the matmul as the paper's
reorder allows).  Same acceptance rule as the SiLU Gated MLP:
|Y_gpu - Y_ref| <= 1e-2 * (|Y_ref| + rms(Y_ref)), elementwise.
"""
import numpy as np
import pytest
import torch

from paper_2606_26344_amd import gmlp
from paper_2606_26344_amd import inputs as I

from test_gpu_parity import _check, _dev

pytestmark = pytest.mark.gpu

VARIANTS = {
    "swiglu": dict(activation="swish", beta=1.702),
    "glu": dict(activation="sigmoid"),
    "rmsnorm": dict(rmsnorm=True, eps=1e-6),
    "rmsnorm_swiglu": dict(activation="swish", beta=0.5, rmsnorm=True, eps=1e-3),
}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    gmlp.library()


def _run(orc, T, D, F, variant, seed, path="auto", rows=None, x_scale=1.0, unit_rms=False):
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=seed, unit_rms_rows=unit_rms)
    if x_scale != 1.0:
        X = I.f32_to_bf16_bits(I.bf16_bits_to_f32(X) * np.float32(x_scale))
    ws = gmlp.Workspace(T, D, F)
    y = gmlp.forward(*[_dev(a) for a in (X, Wg, Wu, Wd)], path=path, workspace=ws, **variant)
    torch.cuda.synchronize()
    rows = np.arange(T) if rows is None else rows
    ref = orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows, **variant)
    return _check(gmlp.to_bf16_bits(y)[rows], ref, "T=%d D=%d F=%d %s %s" % (T, D, F, variant, path))


SHAPES = [(1, 264, 520), (3, 1032, 2056), (8, 264, 264), (17, 520, 1032), (48, 520, 1032),
          (128, 264, 1032), (300, 1032, 2056)]


@pytest.mark.parametrize("name", sorted(VARIANTS))
@pytest.mark.parametrize("T,D,F", SHAPES, ids=["T%dD%dF%d" % s for s in SHAPES])
def test_variant_ragged_shapes(orc, name, T, D, F):
    _run(orc, T, D, F, VARIANTS[name], seed=T * 7 + D, x_scale=3.0)


@pytest.mark.parametrize("name", sorted(VARIANTS))
@pytest.mark.parametrize("T", [100, 150])
def test_variant_paired_gate_up_blocks(orc, name, T):
    # 100 and 150 tokens, 97 column tiles of F: the G and U blocks of a pair
    # (activation and RMSNorm scale applied by the later one).
    assert gmlp.describe(T, 520, 12296)[0][0].endswith(", 2, true, true>")
    _run(orc, T, 520, 12296, VARIANTS[name], seed=77 + T, x_scale=3.0)


@pytest.mark.parametrize("name", sorted(VARIANTS))
@pytest.mark.parametrize("T", [515, 600])
def test_variant_gate_up_token_split(orc, name, T):
    # The gate/up step on a token split (the rest rows through the GEMV
    # kernels at T = 515, through pairs at T = 600), RMSNorm scales included.
    assert len(gmlp.describe(T, 1032, 14344)) == 3
    rows = np.unique(np.concatenate([I.sample_rows(T, 12), np.arange(509, 515)]))
    _run(orc, T, 1032, 14344, VARIANTS[name], seed=50 + T, rows=rows, x_scale=3.0)


@pytest.mark.parametrize("name", sorted(VARIANTS))
@pytest.mark.parametrize("T", [2, 5])
def test_variant_on_the_mfma_path_at_small_T(orc, name, T):
    _run(orc, T, 520, 1032, VARIANTS[name], seed=90 + T, path="mfma", x_scale=0.25)


@pytest.mark.parametrize("name", sorted(VARIANTS))
def test_variant_full_size_decode(orc, name):
    w = I.WORKLOADS["decode"]
    _run(orc, w.T, w.D, w.F, VARIANTS[name], seed=w.seed)


@pytest.mark.parametrize("name", ["rmsnorm", "rmsnorm_swiglu", "glu"])
def test_variant_full_size_prefill_sampled(orc, name):
    w = I.WORKLOADS["large_prefill"]
    _run(orc, w.T, w.D, w.F, VARIANTS[name], seed=w.seed, rows=I.sample_rows(w.T, 32))


def test_variant_gate_up_alone_matches_oracle_h(orc):
    for (T, D, F), path in [((4, 264, 1032), "gemv"), ((40, 520, 264), "auto")]:
        X, Wg, Wu, Wd = I.generate(T, D, F, seed=5)
        v = VARIANTS["rmsnorm_swiglu"]
        ws = gmlp.Workspace(T, D, F)
        h = gmlp.gate_up(_dev(X), _dev(Wg), _dev(Wu), path=path, workspace=ws, **v)
        torch.cuda.synchronize()
        _, H_ref = orc.gated_mlp_rows(X, Wg, Wu, Wd, return_h=True, **v)
        _check(gmlp.to_bf16_bits(h), H_ref, "H %s T=%d" % (path, T))


@pytest.mark.parametrize("T", [1, 6, 64])
def test_silu_variant_is_the_plain_forward_bitwise(T):
    D, F = 1032, 2056
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=8)
    args = [_dev(a) for a in (X, Wg, Wu, Wd)]
    ws = gmlp.Workspace(T, D, F)
    a = gmlp.forward(*args, workspace=ws).clone()
    lib = gmlp.library()
    y = torch.empty_like(a)
    p = gmlp._ptr
    rc = lib.gmlp_forward_variant(p(args[0]), p(args[1]), p(args[2]), p(args[3]), p(y), T, D, F,
                                  gmlp.ACT_SILU, 1.0, 0, 0.0, 0, p(ws.buffer), ws.nbytes,
                                  gmlp._stream(None))
    assert rc == 0, gmlp.last_error()
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), y.view(torch.int16))


@pytest.mark.parametrize("T", [1, 3, 200])
def test_rmsnorm_is_scale_invariant_on_gpu(T):
    """RMSNorm(c x) = RMSNorm(x): scaling X by a power of two (exact in bf16)
    leaves the result unchanged up to the fp32 rounding of the row scale."""
    D, F = 1032, 1032
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=9)
    X8 = I.f32_to_bf16_bits(I.bf16_bits_to_f32(X) * np.float32(8.0))
    outs = []
    for x in (X, X8):
        y = gmlp.forward(_dev(x), _dev(Wg), _dev(Wu), _dev(Wd), workspace=gmlp.Workspace(T, D, F),
                         rmsnorm=True, eps=0.0)
        torch.cuda.synchronize()
        outs.append(I.bf16_bits_to_f32(gmlp.to_bf16_bits(y)).astype(np.float64))
    a, b = outs
    bound = 1e-2 * (np.abs(a) + np.sqrt(np.mean(a ** 2)))
    assert np.all(np.abs(a - b) <= bound)
