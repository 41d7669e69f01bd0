"""Pure-Python scalar brute force of the Gated MLP, for tiny shapes.

TEST INFRASTRUCTURE ONLY.  It is a second, independent spelling of the
definition (Fig. fig:mlp-example, Section 4.2; matmul as a sum of products,
Fig. fig:op-sema; silu(x) = x * sigmoid(x), table tab:nki-ops; RMSNorm,
the equation of Section 2) in plain Python floats and nested loops, used to
pin the C oracle on small inputs.
"""
from __future__ import annotations

import math


def brute_silu(z: float) -> float:
    """x * sigmoid(x) with sigmoid(x) = 1 / (1 + e^-x), overflow-safe."""
    if z >= 0:
        return z * (1.0 / (1.0 + math.exp(-z)))
    e = math.exp(z)
    return z * (e / (1.0 + e))


def brute_sigmoid(z: float) -> float:
    if z >= 0:
        return 1.0 / (1.0 + math.exp(-z))
    e = math.exp(z)
    return e / (1.0 + e)


def brute_gate(g: float, activation: str = "silu", beta: float = 1.0) -> float:
    if activation == "silu":
        return brute_silu(g)
    if activation == "swish":
        return g * brute_sigmoid(beta * g)
    if activation == "sigmoid":
        return brute_sigmoid(g)
    raise ValueError(activation)


def brute_gated_mlp(X, Wg, Wu, Wd, activation="silu", beta=1.0, rmsnorm=False, eps=0.0):
    """X [T][D], Wg [D][F], Wu [D][F], Wd [F][D] as nested lists of floats."""
    T, D, F = len(X), len(Wg), len(Wg[0])
    Y = []
    for t in range(T):
        x = list(X[t])
        if rmsnorm:
            ms = sum(v * v for v in x) / D
            r = 1.0 / math.sqrt(ms + eps)
            x = [v * r for v in x]
        H = []
        for f in range(F):
            g = 0.0
            u = 0.0
            for d in range(D):
                g += x[d] * Wg[d][f]
                u += x[d] * Wu[d][f]
            H.append(brute_gate(g, activation, beta) * u)
        row = []
        for j in range(D):
            acc = 0.0
            for f in range(F):
                acc += H[f] * Wd[f][j]
            row.append(acc)
        Y.append(row)
    return Y


def brute_softmax_matmul(X, Y):
    """Z = softmax(X) Y for X [M][K], Y [K][N] as nested lists of floats:
    exp of every entry, the row sum, the divide, then the matmul (the graph
    of Fig. fig:softmax-matmul-comp-graph (a), Appendix B)."""
    M, K, N = len(X), len(Y), len(Y[0])
    Z = []
    for i in range(M):
        e = [math.exp(X[i][k]) for k in range(K)]
        s = 0.0
        for v in e:
            s += v
        a = [v / s for v in e]
        row = []
        for j in range(N):
            acc = 0.0
            for k in range(K):
                acc += a[k] * Y[k][j]
            row.append(acc)
        Z.append(row)
    return Z
