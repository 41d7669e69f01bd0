"""Pins for the CPU fp64 Softmax+MatMul oracle.

The oracle evaluates the graph of Fig. fig:softmax-matmul-comp-graph (a)
(Appendix B): E = exp(X), S = row sums of E, A = E / S, Z = A Y.  It is tied
here to things other than itself: a library softmax, closed forms (rows of a
softmax sum to one; equal logits give the mean; two logits give the logistic
function; a dominant logit selects a row of Y), invariances the definition
implies (a per-row shift of X, a joint permutation of the contracted axis)
and a pure-Python brute force.  Every pin is a function of an oracle
instance, and the same pins run against copies of the oracle with a planted
mistake; each mutant must fail at least one pin.
"""
from __future__ import annotations

import math
import os
import shutil
import tempfile

import numpy as np
import pytest
from scipy.special import expit, softmax

import oracle
from oracle.softmax_matmul import (
    SOURCE,
    OracleDomainError,
    SoftmaxMatmulOracle,
    build,
    default_oracle,
)


@pytest.fixture(scope="module")
def orc():
    return default_oracle()


def _problem(seed, M, K, N, scale=1.0):
    r = np.random.default_rng(seed)
    return r.standard_normal((M, K)) * scale, r.standard_normal((K, N))


def _close(a, b, atol):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, (a.shape, b.shape)
    err = np.max(np.abs(a - b)) if a.size else 0.0
    assert err <= atol, "max |a - b| = %g > %g" % (err, atol)


# ----------------------------------------------------------------- pins ----
def pin_softmax_matches_library(orc):
    # scipy's softmax (a max-shifted evaluation, a different spelling).
    X, Y = _problem(1, 6, 37, 5, scale=3.0)
    _, A = orc.rows(X, Y, return_softmax=True)
    _close(A, softmax(X, axis=1), 1e-15)


def pin_product_matches_library(orc):
    X, Y = _problem(2, 7, 45, 9, scale=2.0)
    _close(orc.rows(X, Y), softmax(X, axis=1) @ Y, 1e-14)


def pin_rows_of_softmax_sum_to_one(orc):
    # Y = all ones: every output is the row sum of the softmax, exactly 1.
    X, _ = _problem(3, 5, 50, 1, scale=2.0)
    _close(orc.rows(X, np.ones((50, 3))), np.ones((5, 3)), 1e-14)


def pin_equal_logits_give_the_mean(orc):
    # A row of equal logits c: softmax is 1/K everywhere, Z is the mean of the
    # rows of Y, whatever c is.
    K = 24
    _, Y = _problem(4, 1, K, 6)
    X = np.repeat(np.array([[-3.0], [0.0], [5.5]]), K, axis=1)
    _close(orc.rows(X, Y), np.repeat(Y.mean(axis=0)[None, :], 3, axis=0), 1e-14)


def pin_two_logits_are_logistic(orc):
    # K = 2: softmax(x0, x1) = (expit(x0 - x1), expit(x1 - x0)).
    X, Y = _problem(5, 8, 2, 4, scale=3.0)
    p = expit(X[:, 0] - X[:, 1])[:, None]
    q = expit(X[:, 1] - X[:, 0])[:, None]
    _close(orc.rows(X, Y), p * Y[0][None, :] + q * Y[1][None, :], 1e-15)


def pin_dominant_logit_selects_a_row(orc):
    # One logit 40 above the others: Z is that row of Y up to K e^-40 |Y|.
    K = 16
    _, Y = _problem(6, 1, K, 5)
    hot = [3, 0, 15, 7]
    X = np.zeros((len(hot), K))
    for i, k in enumerate(hot):
        X[i, k] = 40.0
    _close(orc.rows(X, Y), Y[hot], K * math.exp(-40.0) * np.abs(Y).max() * 2)


def pin_per_row_shift_invariance(orc):
    # softmax(x + c) = softmax(x) for any constant c per row.
    X, Y = _problem(7, 4, 33, 6)
    shift = np.array([[7.25], [-11.5], [0.0], [30.0]])
    _close(orc.rows(X + shift, Y), orc.rows(X, Y), 1e-13)


def pin_joint_permutation_of_k(orc):
    # Permuting the contracted axis of X and the rows of Y together.
    X, Y = _problem(8, 5, 29, 7)
    perm = np.random.default_rng(9).permutation(29)
    _close(orc.rows(X[:, perm], Y[perm]), orc.rows(X, Y), 1e-14)


def pin_brute_force(orc):
    X, Y = _problem(10, 3, 5, 4, scale=2.0)
    want = np.array(oracle.brute_softmax_matmul(X.tolist(), Y.tolist()))
    _close(orc.rows(X, Y), want, 1e-15)


def pin_row_selection(orc):
    X, Y = _problem(11, 6, 20, 8)
    full = orc.rows(X, Y)
    _close(orc.rows(X, Y, rows=[4, 1, 1, 5]), full[[4, 1, 1, 5]], 0.0)


def pin_bf16_decoding(orc):
    # bf16 bit patterns are the top 16 bits of a binary32: the bf16 entry
    # point must equal the f64 entry point on the decoded values, exactly.
    r = np.random.default_rng(12)
    Xb = (r.standard_normal((4, 40)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    Yb = (r.standard_normal((40, 9)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    dec = lambda b: (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)  # noqa: E731
    assert np.array_equal(orc.rows(Xb, Yb), orc.rows(dec(Xb), dec(Yb)))


def pin_linear_in_y(orc):
    X, Y1 = _problem(13, 3, 18, 4)
    _, Y2 = _problem(14, 3, 18, 4)
    _close(orc.rows(X, 2.0 * Y1 - 0.5 * Y2), 2.0 * orc.rows(X, Y1) - 0.5 * orc.rows(X, Y2), 1e-14)


PINS = [
    pin_softmax_matches_library,
    pin_product_matches_library,
    pin_rows_of_softmax_sum_to_one,
    pin_equal_logits_give_the_mean,
    pin_two_logits_are_logistic,
    pin_dominant_logit_selects_a_row,
    pin_per_row_shift_invariance,
    pin_joint_permutation_of_k,
    pin_brute_force,
    pin_row_selection,
    pin_bf16_decoding,
    pin_linear_in_y,
]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(orc, pin):
    pin(orc)


def test_domain_is_enforced(orc):
    # exp overflows double above ~709.78; a row whose exps all underflow has
    # a zero sum.  Both are reported, not returned as inf or NaN.
    Y = np.ones((3, 2))
    with pytest.raises(OracleDomainError):
        orc.rows(np.array([[0.0, 800.0, 1.0]]), Y)
    with pytest.raises(OracleDomainError):
        orc.rows(np.array([[-800.0, -900.0, -1000.0]]), Y)
    # Large but representable logits are inside the domain.
    Z = orc.rows(np.array([[700.0, 0.0, 0.0]]), np.eye(3))
    assert Z[0, 0] == 1.0


def test_empty_row_list(orc):
    X, Y = _problem(15, 4, 8, 3)
    assert orc.rows(X, Y, rows=[]).shape == (0, 3)


def test_bad_row_index(orc):
    X, Y = _problem(16, 4, 8, 3)
    with pytest.raises(RuntimeError):
        orc.rows(X, Y, rows=[4])


# ------------------------------------------------------------- mutants ----
# (description, snippet of softmax_matmul_oracle.c, replacement); each
# snippet occurs exactly once in the source.
MUTANTS = [
    ("divide dropped (unnormalised exp times Y)",
     "a[k] = a[k] / s;",
     "a[k] = a[k];"),
    ("exp dropped",
     "a[k] = exp(LD(X, t * K + k));",
     "a[k] = LD(X, t * K + k);"),
    ("first term of the row sum dropped",
     "s += a[k];",
     "s += k ? a[k] : 0.0;"),
    ("normalised by the first exp instead of the sum",
     "a[k] = a[k] / s;",
     "a[k] = a[k] / a[0];"),
    ("rows of Y read in reverse",
     "z[j] += ak * LD(Y, k * N + j);",
     "z[j] += ak * LD(Y, (K - 1 - k) * N + j);"),
    ("columns of Y read in reverse",
     "z[j] += ak * LD(Y, k * N + j);",
     "z[j] += ak * LD(Y, k * N + (N - 1 - j));"),
    ("always row 0 of X",
     "a[k] = exp(LD(X, t * K + k));",
     "a[k] = exp(LD(X, k));"),
    ("last term of the matmul dropped",
     "double ak = a[k];",
     "double ak = k + 1 < K ? a[k] : 0.0;"),
    ("bf16 decoded with the wrong shift",
     "uint32_t u = (uint32_t)p[i] << 16;",
     "uint32_t u = (uint32_t)p[i] << 15;"),
    ("exp of the negated logits",
     "a[k] = exp(LD(X, t * K + k));",
     "a[k] = exp(-LD(X, t * K + k));"),
]


def _run_pins(orc):
    failed = []
    for pin in PINS:
        try:
            pin(orc)
        except (AssertionError, OracleDomainError, RuntimeError):
            failed.append(pin.__name__)
    return failed


def test_pins_pass_on_the_oracle(orc):
    assert _run_pins(orc) == []


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc to build mutants")
@pytest.mark.parametrize("mutant", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(mutant):
    desc, old, new = mutant
    src = open(SOURCE).read()
    assert src.count(old) == 1, "mutant snippet no longer matches the oracle source: %r" % old
    with tempfile.TemporaryDirectory() as tmp:
        path = os.path.join(tmp, "mutant.c")
        with open(path, "w") as fh:
            fh.write(src.replace(old, new))
        lib = build(path, os.path.join(tmp, "libmutant.so"))
        failed = _run_pins(SoftmaxMatmulOracle(lib))
    assert failed, "no pin detects the planted mistake: %s" % desc
