"""Pins for the CPU fp64 oracle.

The oracle is trusted only because it is tied here to things other than
itself: closed forms, identities, library routines, a pure-Python brute force
and a hand-built example with an exact answer.  Each pin is a function of an
oracle instance, so the same pins are also run against copies of the oracle
with a planted mistake (compiled from a mutated source); every such mutant
must fail at least one pin, which shows the pins can see that kind of error.

Definitions pinned (from the paper):
  * the Gated MLP graph, Fig. fig:mlp-example (Section 4.1);
  * matmul as a sum of products, Fig. fig:op-sema (Section 4.2.1);
  * silu(x) = x * sigmoid(x), table tab:nki-ops (Section 5.1);
  * the illegal "silu past multiply" swap (Section 5.1, Examples) is one of
    the planted mutants;
  * the variants: gate activations swish_beta(g) = g * sigmoid(beta g) and
    sigmoid(g) (the paper's SwiGLU / GLU benchmarks, Section 6.1, usual
    definitions), and RMSNorm in front (the RMSNorm equation, Section 2).
"""
from __future__ import annotations

import math
import os
import shutil
import tempfile
from fractions import Fraction

import numpy as np
import pytest
from scipy.special import expit

import oracle
from oracle.oracle import Oracle, build, SOURCE

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _rand_problem(seed, T, D, F, scale=1.0):
    r = _rng(seed)
    X = r.standard_normal((T, D)) * scale
    Wg = r.standard_normal((D, F)) / math.sqrt(D)
    Wu = r.standard_normal((D, F)) / math.sqrt(D)
    Wd = r.standard_normal((F, D)) / math.sqrt(F)
    return X, Wg, Wu, Wd


def _library_gated_mlp(X, Wg, Wu, Wd):
    """Library spelling: numpy matmul and scipy's logistic sigmoid."""
    G = X @ Wg
    U = X @ Wu
    return (G * expit(G) * U) @ Wd


def _close(a, b, rtol, atol=0.0):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    err = np.abs(a - b)
    bound = atol + rtol * np.abs(b)
    return bool(np.all(err <= bound)), float(np.max(err - bound)) if err.size else 0.0


# ---------------------------------------------------------------- pins ----

def pin_silu_zero(orc):
    assert orc.silu(0.0) == 0.0


def pin_silu_logit_points(orc):
    """sigmoid(ln(p/(1-p))) = p exactly, so silu(ln(p/(1-p))) = p ln(p/(1-p))."""
    with open(os.path.join(GOLDEN, "silu_logit_points.txt")) as fh:
        ps = [Fraction(line.strip()) for line in fh if line.strip() and not line.startswith("#")]
    assert len(ps) >= 8
    for p in ps:
        x = math.log(p / (1 - p))
        want = float(p) * x
        got = orc.silu(x)
        # x itself carries a rounding error of about |x| eps, which moves
        # sigmoid(x) by (1 - p) |x| eps relative; allow that plus a few ulps.
        tol = 2.3e-16 * (4.0 + 2.0 * abs(x)) * abs(want)
        assert abs(got - want) <= tol, (p, got, want)


def pin_silu_odd_part(orc):
    """sigmoid(x) + sigmoid(-x) = 1 implies silu(x) - silu(-x) = x."""
    xs = np.concatenate([np.linspace(-30, 30, 241), [1e-8, 0.5, 2.0, 7.25, 19.0]])
    for x in xs:
        got = orc.silu(x) - orc.silu(-x)
        assert abs(got - x) <= 4e-16 * max(1.0, abs(x)), (x, got)


def pin_silu_library(orc):
    """Against x * scipy.special.expit(x) (library logistic function)."""
    xs = np.concatenate([np.linspace(-40, 40, 801), [-700.0, -100.0, 100.0, 700.0]])
    got = orc.silu(xs)
    want = xs * expit(xs)
    ok, worst = _close(got, want, 1e-14, 1e-300)
    assert ok, worst


def pin_silu_extremes(orc):
    """silu(x) -> x for large x, -> 0 (no NaN, no overflow) for very negative x."""
    assert orc.silu(60.0) == 60.0
    v = orc.silu(-40.0)
    assert abs(v - (-40.0 * math.exp(-40.0))) <= 1e-15 * 40.0 * math.exp(-40.0)
    for x in (-745.0, -1000.0, -1e300):
        v = orc.silu(x)
        assert not math.isnan(v) and v <= 0.0 and abs(v) < 1e-300


def pin_brute_force_f64(orc):
    """C oracle vs the pure-Python triple loop on tiny random shapes."""
    for seed, (T, D, F) in enumerate([(1, 1, 1), (1, 2, 3), (2, 3, 2), (3, 5, 7),
                                      (3, 8, 8), (2, 7, 4), (1, 8, 1)]):
        X, Wg, Wu, Wd = _rand_problem(100 + seed, T, D, F, scale=1.5)
        got = orc.gated_mlp_rows(X, Wg, Wu, Wd)
        want = np.array(oracle.brute_gated_mlp(X.tolist(), Wg.tolist(), Wu.tolist(), Wd.tolist()))
        ok, worst = _close(got, want, 1e-12, 1e-14)
        assert ok, (T, D, F, worst)


def pin_brute_force_bf16(orc):
    """bf16 bit-pattern inputs: decoded exactly, then as the brute force."""
    from paper_2606_26344_amd.inputs import bf16_bits_to_f32, f32_to_bf16_bits

    for seed, (T, D, F) in enumerate([(2, 8, 8), (3, 4, 6), (1, 8, 16)]):
        X, Wg, Wu, Wd = [f32_to_bf16_bits(a.astype(np.float32))
                         for a in _rand_problem(200 + seed, T, D, F)]
        got = orc.gated_mlp_rows(X, Wg, Wu, Wd)
        dec = [bf16_bits_to_f32(a).astype(np.float64).tolist() for a in (X, Wg, Wu, Wd)]
        want = np.array(oracle.brute_gated_mlp(*dec))
        ok, worst = _close(got, want, 1e-12, 1e-14)
        assert ok, (T, D, F, worst)


def pin_zero_gate_or_up(orc):
    """silu(0) = 0 and H is linear in U: Wg = 0 or Wu = 0 gives Y = 0 exactly."""
    X, Wg, Wu, Wd = _rand_problem(3, 4, 12, 20)
    assert np.all(orc.gated_mlp_rows(X, np.zeros_like(Wg), Wu, Wd) == 0.0)
    assert np.all(orc.gated_mlp_rows(X, Wg, np.zeros_like(Wu), Wd) == 0.0)
    assert np.all(orc.gated_mlp_rows(np.zeros_like(X), Wg, Wu, Wd) == 0.0)


def pin_linearity(orc):
    """Y is linear in Wd and in Wu (for fixed X, Wg)."""
    X, Wg, Wu, Wd = _rand_problem(4, 3, 10, 14)
    _, _, Wu2, Wd2 = _rand_problem(5, 3, 10, 14)
    a, b = 0.75, -1.25
    y1 = orc.gated_mlp_rows(X, Wg, Wu, a * Wd + b * Wd2)
    y2 = a * orc.gated_mlp_rows(X, Wg, Wu, Wd) + b * orc.gated_mlp_rows(X, Wg, Wu, Wd2)
    ok, worst = _close(y1, y2, 1e-12, 1e-13)
    assert ok, worst
    y1 = orc.gated_mlp_rows(X, Wg, a * Wu + b * Wu2, Wd)
    y2 = a * orc.gated_mlp_rows(X, Wg, Wu, Wd) + b * orc.gated_mlp_rows(X, Wg, Wu2, Wd)
    ok, worst = _close(y1, y2, 1e-12, 1e-13)
    assert ok, worst


def pin_one_hot_rows(orc):
    """X[t] = e_d selects row d of Wg and Wu: Y[t] = (silu(Wg[d]) * Wu[d]) Wd."""
    D, F = 6, 9
    _, Wg, Wu, Wd = _rand_problem(6, 1, D, F, scale=1.0)
    Wg = Wg * 3.0
    X = np.eye(D)
    got = orc.gated_mlp_rows(X, Wg, Wu, Wd)
    for d in range(D):
        g = Wg[d]
        want = (g * expit(g) * Wu[d]) @ Wd
        ok, worst = _close(got[d], want, 1e-13, 1e-15)
        assert ok, (d, worst)


def pin_permutations(orc):
    """Permuting the F axis of Wg, Wu and Wd together leaves Y unchanged;
    evaluating a permuted list of rows permutes the rows of Y."""
    X, Wg, Wu, Wd = _rand_problem(7, 5, 8, 11)
    pi = _rng(8).permutation(11)
    y = orc.gated_mlp_rows(X, Wg, Wu, Wd)
    yp = orc.gated_mlp_rows(X, Wg[:, pi], Wu[:, pi], Wd[pi, :])
    ok, worst = _close(yp, y, 1e-12, 1e-14)
    assert ok, worst
    rows = [4, 0, 3, 3, 1]
    ok, worst = _close(orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows), y[rows], 0.0, 0.0)
    assert ok, worst


def pin_library_composite(orc):
    """Whole path against numpy matmul + scipy expit at a moderate size."""
    for seed, (T, D, F) in enumerate([(5, 96, 200), (2, 33, 70), (7, 64, 64)]):
        X, Wg, Wu, Wd = _rand_problem(300 + seed, T, D, F, scale=2.0)
        got = orc.gated_mlp_rows(X, Wg, Wu, Wd)
        want = _library_gated_mlp(X, Wg, Wu, Wd)
        scale = np.sqrt(np.mean(want ** 2))
        ok, worst = _close(got, want, 1e-12, 1e-13 * scale)
        assert ok, (T, D, F, worst)


def _read_logq_example():
    vals = {}
    with open(os.path.join(GOLDEN, "gated_mlp_logq.txt")) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, rhs = (s.strip() for s in line.split("=", 1))
            vals[key] = [[Fraction(tok) for tok in row.split()] for row in rhs.split(";")]
    return vals


def pin_golden_logq(orc):
    """Hand-built example with G = ln(q), so sigmoid(G) = q / (1 + q) exactly."""
    ex = _read_logq_example()
    X, A, Wu, Wd = ex["X"], ex["A"], ex["Wu"], ex["Wd"]
    T, D, F = len(X), len(A), len(A[0])
    want = [[0.0] * D for _ in range(T)]
    for t in range(T):
        for f in range(F):
            q = Fraction(1)
            for d in range(D):
                q *= A[d][f] ** int(X[t][d])
            u = sum(X[t][d] * Wu[d][f] for d in range(D))
            h = math.log(q) * float(q / (1 + q) * u)
            for j in range(D):
                want[t][j] += h * float(Wd[f][j])
    Xf = np.array([[float(v) for v in row] for row in X])
    Wg = np.array([[math.log(v) for v in row] for row in A])
    got = orc.gated_mlp_rows(Xf, Wg, np.array(Wu, dtype=float), np.array(Wd, dtype=float))
    ok, worst = _close(got, np.array(want), 1e-13, 1e-14)
    assert ok, (got, want, worst)


def pin_bf16_path_matches_f64_path(orc):
    """The bf16 entry point equals the f64 one on the exactly decoded values."""
    from paper_2606_26344_amd.inputs import bf16_bits_to_f32, generate

    X, Wg, Wu, Wd = generate(9, 40, 72, seed=3)
    a = orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=[0, 4, 8])
    b = orc.gated_mlp_rows(*[bf16_bits_to_f32(m).astype(np.float64) for m in (X, Wg, Wu, Wd)],
                           rows=[0, 4, 8])
    assert np.array_equal(a, b)


def pin_down_step_alone(orc):
    """The down projection alone: one-hot rows of H select rows of Wd, and
    random bf16 data agrees with numpy's matmul."""
    from paper_2606_26344_amd.inputs import bf16_bits_to_f32, f32_to_bf16_bits

    F, D = 24, 16
    Wd = f32_to_bf16_bits(_rng(11).standard_normal((F, D)).astype(np.float32))
    eye = f32_to_bf16_bits(np.eye(F, dtype=np.float32))
    got = orc.down_rows(eye, Wd)
    assert np.array_equal(got, bf16_bits_to_f32(Wd).astype(np.float64))
    H = f32_to_bf16_bits(_rng(12).standard_normal((5, F)).astype(np.float32))
    want = bf16_bits_to_f32(H).astype(np.float64) @ bf16_bits_to_f32(Wd).astype(np.float64)
    ok, worst = _close(orc.down_rows(H, Wd, rows=[4, 1]), want[[4, 1]], 1e-13, 1e-14)
    assert ok, worst


PINS = [
    pin_silu_zero,
    pin_silu_logit_points,
    pin_silu_odd_part,
    pin_silu_library,
    pin_silu_extremes,
    pin_brute_force_f64,
    pin_brute_force_bf16,
    pin_zero_gate_or_up,
    pin_linearity,
    pin_one_hot_rows,
    pin_permutations,
    pin_library_composite,
    pin_golden_logq,
    pin_bf16_path_matches_f64_path,
    pin_down_step_alone,
]


# ---------------------------------------------------------------- variants ----
def _logit_ps():
    ps = []
    with open(os.path.join(GOLDEN, "silu_logit_points.txt")) as fh:
        for line in fh:
            line = line.split("#")[0].strip()
            if line:
                ps.append(Fraction(line))
    return ps


def pin_sigmoid_logit_points(orc):
    # sigmoid(ln(p / (1 - p))) = p exactly; the GLU gate.
    for p in _logit_ps():
        x = math.log(p / (1 - p))
        want = float(p)
        got = orc.gate(x, "sigmoid")
        assert abs(got - want) <= 2.3e-16 * (4 + 2 * abs(x)) * abs(want), (p, got)
        assert orc.sigmoid(x) == got


def pin_swish_logit_points(orc):
    # beta * x = ln(p / (1 - p))  =>  swish_beta(x) = x * p.
    for beta in (0.5, 1.702, 3.0):
        for p in _logit_ps():
            x = math.log(p / (1 - p)) / beta
            want = x * float(p)
            got = orc.gate(x, "swish", beta)
            assert abs(got - want) <= 2.3e-16 * (6 + 2 * abs(beta * x)) * abs(want), (beta, p, got)


def pin_swish_beta_zero_is_bilinear(orc):
    # swish_0(g) = g / 2: Y = ((X Wg) / 2 * (X Wu)) Wd, a library matmul.
    X, Wg, Wu, Wd = _rand_problem(41, 3, 16, 24)
    want = (0.5 * (X @ Wg) * (X @ Wu)) @ Wd
    got = orc.gated_mlp_rows(X, Wg, Wu, Wd, activation="swish", beta=0.0)
    ok, worst = _close(got, want, 1e-12, 1e-14)
    assert ok, worst


def pin_swish_large_beta_is_relu(orc):
    # beta -> inf: swish_beta(g) -> max(g, 0) (error below g e^{-beta |g|}).
    X, Wg, Wu, Wd = _rand_problem(42, 3, 16, 24)
    G = X @ Wg
    assert np.min(np.abs(G)) > 1e-3
    want = (np.maximum(G, 0.0) * (X @ Wu)) @ Wd
    got = orc.gated_mlp_rows(X, Wg, Wu, Wd, activation="swish", beta=1e6)
    ok, worst = _close(got, want, 1e-10, 1e-12)
    assert ok, worst


def pin_glu_library(orc):
    # sigmoid gate against numpy matmul and scipy's logistic function.
    X, Wg, Wu, Wd = _rand_problem(43, 4, 32, 40, scale=2.0)
    want = (expit(X @ Wg) * (X @ Wu)) @ Wd
    got = orc.gated_mlp_rows(X, Wg, Wu, Wd, activation="sigmoid")
    ok, worst = _close(got, want, 1e-12, 1e-13)
    assert ok, worst


def pin_glu_zero_gate_halves_up(orc):
    # Wg = 0: sigmoid(0) = 1/2 exactly, so Y = ((X Wu) / 2) Wd.
    X, Wg, Wu, Wd = _rand_problem(44, 3, 16, 24)
    want = (0.5 * (X @ Wu)) @ Wd
    got = orc.gated_mlp_rows(X, np.zeros_like(Wg), Wu, Wd, activation="sigmoid")
    ok, worst = _close(got, want, 1e-12, 1e-14)
    assert ok, worst


def pin_variants_brute_force(orc):
    X, Wg, Wu, Wd = _rand_problem(45, 2, 5, 7, scale=1.5)
    lists = [a.tolist() for a in (X, Wg, Wu, Wd)]
    for kw in ({"activation": "swish", "beta": 1.7}, {"activation": "sigmoid"},
               {"rmsnorm": True, "eps": 1e-3}, {"activation": "swish", "beta": 0.3,
                                                "rmsnorm": True, "eps": 0.25}):
        want = np.array(oracle.brute_gated_mlp(*lists, **kw))
        got = orc.gated_mlp_rows(X, Wg, Wu, Wd, **kw)
        ok, worst = _close(got, want, 1e-12, 1e-14)
        assert ok, (kw, worst)


def pin_rmsnorm_unit_rows_are_unchanged(orc):
    # Rows of +-1 have mean(x^2) = 1 exactly: with eps = 0 RMSNorm is the
    # identity, so the result equals the plain Gated MLP bit for bit.
    r = _rng(46)
    X = np.where(r.standard_normal((4, 32)) > 0, 1.0, -1.0)
    _, Wg, Wu, Wd = _rand_problem(46, 4, 32, 24)
    plain = orc.gated_mlp_rows(X, Wg, Wu, Wd)
    normed = orc.gated_mlp_rows(X, Wg, Wu, Wd, rmsnorm=True, eps=0.0)
    assert np.array_equal(plain, normed)


def pin_rmsnorm_scale_invariant(orc):
    # RMSNorm(c x) = RMSNorm(x) for c > 0 when eps = 0.
    X, Wg, Wu, Wd = _rand_problem(47, 3, 32, 24)
    a = orc.gated_mlp_rows(X, Wg, Wu, Wd, rmsnorm=True, eps=0.0)
    b = orc.gated_mlp_rows(X * 37.0, Wg, Wu, Wd, rmsnorm=True, eps=0.0)
    ok, worst = _close(b, a, 1e-13, 1e-15)
    assert ok, worst
    assert not np.allclose(a, orc.gated_mlp_rows(X, Wg, Wu, Wd), rtol=1e-3)


def pin_rmsnorm_closed_form_eps(orc):
    # A row of equal values a: mean(x^2) = a^2, so RMSNorm gives
    # a / sqrt(a^2 + eps); with a = 1, eps = 3 that is exactly 1/2.
    _, Wg, Wu, Wd = _rand_problem(48, 1, 16, 24)
    X = np.ones((1, 16))
    want = orc.gated_mlp_rows(0.5 * X, Wg, Wu, Wd)
    got = orc.gated_mlp_rows(X, Wg, Wu, Wd, rmsnorm=True, eps=3.0)
    assert np.array_equal(got, want)


PINS += [
    pin_sigmoid_logit_points,
    pin_swish_logit_points,
    pin_swish_beta_zero_is_bilinear,
    pin_swish_large_beta_is_relu,
    pin_glu_library,
    pin_glu_zero_gate_halves_up,
    pin_variants_brute_force,
    pin_rmsnorm_unit_rows_are_unchanged,
    pin_rmsnorm_scale_invariant,
    pin_rmsnorm_closed_form_eps,
]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(orc, pin):
    pin(orc)


def test_brute_force_handles_large_negative_gate():
    assert oracle.brute_silu(-1000.0) == 0.0 or oracle.brute_silu(-1000.0) == -0.0
    assert oracle.brute_silu(0.0) == 0.0


# ------------------------------------------------------------- mutants ----
# (description, snippet of gmlp_oracle.c, replacement).  Each snippet must
# occur exactly once in the source.
MUTANTS = [
    ("silu moved past the multiply (the illegal swap of Section 5.1)",
     "h[f_lo + j] = gmlp_oracle_gate(g[j], act, beta) * u[j];",
     "h[f_lo + j] = gmlp_oracle_gate(g[j] * u[j], act, beta);"),
    ("gate and up swapped",
     "h[f_lo + j] = gmlp_oracle_gate(g[j], act, beta) * u[j];",
     "h[f_lo + j] = gmlp_oracle_gate(u[j], act, beta) * g[j];"),
    ("gate activation dropped",
     "h[f_lo + j] = gmlp_oracle_gate(g[j], act, beta) * u[j];",
     "h[f_lo + j] = g[j] * u[j];"),
    ("sigmoid argument sign flipped",
     "return z / (1.0 + exp(-z));",
     "return z / (1.0 + exp(z));"),
    ("negative branch of silu wrong",
     "return z * e / (1.0 + e);",
     "return z * e;"),
    ("Wd read transposed",
     "y[j] += hf * LD(Wd, f * D + j);",
     "y[j] += hf * LD(Wd, j * F + f);"),
    ("Wg read transposed",
     "g[j] += xd * LD(Wg, d * F + f_lo + j);",
     "g[j] += xd * LD(Wg, (f_lo + j) * D + d);"),
    ("last term of the d reduction dropped",
     "for (int64_t d = 0; d < D; ++d) {",
     "for (int64_t d = 0; d + 1 < D; ++d) {"),
    ("requested row list ignored",
     "xr[d] = LD(X, t * D + d);",
     "xr[d] = LD(X, r * D + d);"),
    ("bf16 decoded with the wrong shift",
     "uint32_t u = (uint32_t)p[i] << 16;",
     "uint32_t u = (uint32_t)p[i] << 15;"),
    ("swish ignores beta",
     "case ORACLE_ACT_SWISH: return g * gmlp_oracle_sigmoid(beta * g);",
     "case ORACLE_ACT_SWISH: return g * gmlp_oracle_sigmoid(g);"),
    ("GLU gate computes silu",
     "default: return gmlp_oracle_sigmoid(g);",
     "default: return gmlp_oracle_silu(g);"),
    ("sigmoid sign flipped",
     "return 1.0 / (1.0 + exp(-z));",
     "return 1.0 / (1.0 + exp(z));"),
    ("sigmoid negative branch wrong",
     "return e / (1.0 + e);",
     "return 1.0 / (1.0 + e);"),
    ("RMSNorm eps dropped",
     "double inv = 1.0 / sqrt(ss / (double)D + eps);",
     "double inv = 1.0 / sqrt(ss / (double)D);"),
    ("RMSNorm sum instead of mean",
     "double inv = 1.0 / sqrt(ss / (double)D + eps);",
     "double inv = 1.0 / sqrt(ss + eps);"),
    ("RMSNorm scale not applied",
     "xr[d] = xr[d] * inv;",
     "xr[d] = xr[d] * 1.0;"),
]


def _run_pins(orc):
    failed = []
    for pin in PINS:
        try:
            pin(orc)
        except AssertionError:
            failed.append(pin.__name__)
    return failed


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
        failed = _run_pins(Oracle(lib))
    assert failed, "no pin detects the planted mistake: %s" % desc
