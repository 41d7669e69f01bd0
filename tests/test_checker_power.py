"""Power of the parity rule at the five workloads' full sizes (CPU only).

The GPU parity tests accept an output when every element satisfies
|Y - Y_ref| <= 1e-2 (|Y_ref| + rms(Y_ref)) against the fp64 oracle.  This file
shows, without building any broken kernel, that the rule rejects the mistakes
a kernel of this path could plausibly make, at the real shapes and on the
same sampled rows the GPU tests check:

  * the activation applied after the multiply, silu(g u): the illegal move
    of silu past the multiply (Section 5.1, equivalence examples);
  * the gate and up projections swapped, silu(u) g;
  * the activation dropped, g u;
  * one k-tile (32 rows of D) missing from the gate/up sums;
  * one k-tile (64 rows of F) missing from the down sum;
  * G and U rounded to bf16 before the activation (an extra rounding step);
  * H converted to fp16 but stored where the down step reads bf16 (the
    wrong conversion instruction in the epilogue).

The GPU's numerics are emulated with numpy: float32 products and sums, H
rounded once to bf16 (round to nearest even), Y rounded to bf16.  That
emulation must pass; so must H kept in fp16 end to end, stored and read as
fp16 (three more mantissa bits than the prescribed bf16: more accurate, not
a mistake, so no tolerance could reject it; fp16 bits read as bf16 are a
mistake and are rejected).  H truncated to bf16
instead of rounded to nearest also stays within the rule (its error is at
most one bf16 step, like rounding's); the GPU test
test_h_is_rounded_once_to_nearest_even pins the rounding mode instead.
"""
import numpy as np
import pytest

from paper_2606_26344_amd import inputs as I

TOL = 1e-2
# Rows checked per workload: all of them where the oracle is quick, else
# sampled rows as in the GPU tests.
ROWS = {"tiny": None, "decode": None, "small_batch": 16, "prefill": 4, "large_prefill": 4}


def passes(got, ref):
    """The GPU tests' acceptance rule."""
    got = np.asarray(got, dtype=np.float64)
    bound = TOL * (np.abs(ref) + np.sqrt(np.mean(ref ** 2)))
    return bool(np.all(np.isfinite(got)) and np.all(np.abs(got - ref) <= bound))


def worst_ratio(got, ref):
    bound = TOL * (np.abs(ref) + np.sqrt(np.mean(ref ** 2)))
    return float(np.max(np.abs(np.asarray(got, np.float64) - ref) / bound))


def bf16(a):
    return I.bf16_bits_to_f32(I.f32_to_bf16_bits(np.asarray(a, np.float32)))


def bf16_truncated(a):
    bits = (np.ascontiguousarray(a, np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    return I.bf16_bits_to_f32(bits)


def silu(z):
    return z / (np.float32(1) + np.exp(-z))


@pytest.fixture(scope="module", params=list(ROWS))
def emulated(request, orc):
    """Oracle rows and the float32 pieces of the emulation for one workload."""
    name = request.param
    w = I.WORKLOADS[name]
    X, Wg, Wu, Wd = I.generate(w.T, w.D, w.F, seed=w.seed, unit_rms_rows=w.unit_rms_rows)
    rows = np.arange(w.T) if ROWS[name] is None else I.sample_rows(w.T, ROWS[name])
    ref = orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows)
    x = I.bf16_bits_to_f32(X[rows])
    del X
    wg = I.bf16_bits_to_f32(Wg)
    del Wg
    wu = I.bf16_bits_to_f32(Wu)
    del Wu
    wd = I.bf16_bits_to_f32(Wd)
    del Wd
    G, U = x @ wg, x @ wu
    k0 = 32 * (w.D // 64)  # a k-tile in the middle of D
    G_drop = G - x[:, k0:k0 + 32] @ wg[k0:k0 + 32]
    U_drop = U - x[:, k0:k0 + 32] @ wu[k0:k0 + 32]
    del wg, wu
    return dict(name=name, ref=ref, G=G, U=U, G_drop=G_drop, U_drop=U_drop, wd=wd, F=w.F)


def _down(e, H):
    """Y = bf16(bf16(H) Wd) as the down kernel computes it."""
    return bf16(bf16(H) @ e["wd"])


def test_emulated_kernel_numerics_pass(emulated):
    e = emulated
    Y = _down(e, silu(e["G"]) * e["U"])
    print("%s: emulated kernel, worst ratio %.3f" % (e["name"], worst_ratio(Y, e["ref"])))
    assert passes(Y, e["ref"])


def test_more_accurate_or_truncated_h_is_within_the_rule(emulated):
    e = emulated
    H = silu(e["G"]) * e["U"]
    fp16 = bf16(H.astype(np.float16).astype(np.float32) @ e["wd"])
    trunc = bf16(bf16_truncated(H) @ e["wd"])
    assert passes(fp16, e["ref"]), worst_ratio(fp16, e["ref"])
    assert passes(trunc, e["ref"]), worst_ratio(trunc, e["ref"])


MISTAKES = {
    "silu(g*u): activation moved past the multiply": lambda e: _down(e, silu(e["G"] * e["U"])),
    "gate and up swapped": lambda e: _down(e, silu(e["U"]) * e["G"]),
    "activation dropped": lambda e: _down(e, e["G"] * e["U"]),
    "one gate/up k-tile dropped": lambda e: _down(e, silu(e["G_drop"]) * e["U_drop"]),
    "one down k-tile dropped": lambda e: _drop_down_tile(e),
    "G and U rounded to bf16 before the activation": lambda e: _down(e, silu(bf16(e["G"])) * bf16(e["U"])),
    "H stored as fp16 bits, read as bf16": lambda e: _fp16_bits_read_as_bf16(e),
}


def _fp16_bits_read_as_bf16(e):
    bits = (silu(e["G"]) * e["U"]).astype(np.float16).view(np.uint16)
    return bf16(I.bf16_bits_to_f32(bits) @ e["wd"])


def _drop_down_tile(e):
    H = bf16(silu(e["G"]) * e["U"])
    f0 = 64 * (e["F"] // 128)
    return bf16(H @ e["wd"] - H[:, f0:f0 + 64] @ e["wd"][f0:f0 + 64])


@pytest.mark.parametrize("mistake", list(MISTAKES))
def test_kernel_class_mistake_fails_the_rule(emulated, mistake):
    e = emulated
    Y = MISTAKES[mistake](e)
    r = worst_ratio(Y, e["ref"])
    print("%s, %s: worst ratio %.2f" % (e["name"], mistake, r))
    assert not passes(Y, e["ref"]), "%s passed the rule at %s (ratio %.3f)" % (mistake, e["name"], r)
