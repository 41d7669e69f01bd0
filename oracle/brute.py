"""Pure-Python scalar brute force of the SiLU Gated MLP, for tiny shapes.

TEST INFRASTRUCTURE ONLY.  It is a second, independent spelling of the
definition (Fig. fig:mlp-example, Section 4.1; matmul as a sum of products,
Fig. fig:op-sema; silu(x) = x * sigmoid(x), table tab:nki-ops) in plain
Python floats and nested loops, used to pin the C oracle on small inputs.
"""
from __future__ import annotations

import math


def brute_silu(z: float) -> float:
    """x * sigmoid(x) with sigmoid(x) = 1 / (1 + e^-x), overflow-safe."""
    if z >= 0:
        return z * (1.0 / (1.0 + math.exp(-z)))
    e = math.exp(z)
    return z * (e / (1.0 + e))


def brute_gated_mlp(X, Wg, Wu, Wd):
    """X [T][D], Wg [D][F], Wu [D][F], Wd [F][D] as nested lists of floats."""
    T, D, F = len(X), len(Wg), len(Wg[0])
    Y = []
    for t in range(T):
        H = []
        for f in range(F):
            g = 0.0
            u = 0.0
            for d in range(D):
                g += X[t][d] * Wg[d][f]
                u += X[t][d] * Wu[d][f]
            H.append(brute_silu(g) * u)
        row = []
        for j in range(D):
            acc = 0.0
            for f in range(F):
                acc += H[f] * Wd[f][j]
            row.append(acc)
        Y.append(row)
    return Y
