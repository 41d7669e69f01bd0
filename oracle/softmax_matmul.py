"""ctypes wrapper around the C fp64 oracle for Softmax+MatMul
(``softmax_matmul_oracle.c``).

TEST INFRASTRUCTURE ONLY: nothing on the product path may import this module.

The oracle evaluates the graph of Fig. fig:softmax-matmul-comp-graph (a)
(Appendix B): exp, a row sum, a divide, then the matmul, i.e.
Z = softmax(X) Y with the softmax along the contracted axis, in IEEE double
precision on a chosen subset of rows of X.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

from .oracle import build as _compile

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "softmax_matmul_oracle.c")
LIBRARY = os.path.join(HERE, "libsmm_oracle.so")

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_INT = ctypes.c_int

# Return codes of the C entry points.
ERRORS = {1: "bad argument", 2: "row index out of range", 3: "allocation failure",
          4: "a row is outside the oracle's domain (exp or its row sum not finite and nonzero)"}


class OracleDomainError(ValueError):
    """A requested row has exp(x) or its sum outside double precision."""


def build(source: str = SOURCE, output: str = LIBRARY, extra_flags: Sequence[str] = ()) -> str:
    """Compile ``source`` into the shared library ``output`` with gcc."""
    return _compile(source, output, extra_flags)


class SoftmaxMatmulOracle:
    """One loaded copy of the Softmax+MatMul oracle library."""

    def __init__(self, path: str = LIBRARY):
        self.path = path
        lib = ctypes.CDLL(path)
        for name in ("smm_oracle_rows_bf16", "smm_oracle_rows_f64"):
            fn = getattr(lib, name)
            fn.argtypes = [_P, _P, _I64, _I64, _I64, _P, _I64, _P, _P, _INT]
            fn.restype = _INT
        self.lib = lib

    def rows(self, X, Y, rows: Optional[Sequence[int]] = None, threads: int = 0,
             return_softmax: bool = False):
        """Rows of Z = softmax(X) Y in double precision.

        X [M, K] and Y [K, N]: both ``uint16`` (bf16 bit patterns, decoded
        exactly) or both floating point (converted to float64).  ``rows``
        selects rows of X (default: all).  Returns Z [len(rows), N] (and the
        softmax A [len(rows), K] if ``return_softmax``).
        """
        X = np.asarray(X)
        Y = np.asarray(Y)
        if X.dtype == np.uint16 and Y.dtype == np.uint16:
            fn = self.lib.smm_oracle_rows_bf16
            X = np.ascontiguousarray(X)
            Y = np.ascontiguousarray(Y)
        elif X.dtype != np.uint16 and Y.dtype != np.uint16:
            fn = self.lib.smm_oracle_rows_f64
            X = np.ascontiguousarray(X, dtype=np.float64)
            Y = np.ascontiguousarray(Y, dtype=np.float64)
        else:
            raise TypeError("mixing bf16 bit patterns and floating-point inputs")
        if X.ndim != 2 or Y.ndim != 2 or Y.shape[0] != X.shape[1]:
            raise ValueError("shape mismatch: X %s Y %s" % (X.shape, Y.shape))
        M, K = X.shape
        N = Y.shape[1]
        rows_arr = (np.arange(M, dtype=np.int64) if rows is None
                    else np.ascontiguousarray(np.asarray(rows, dtype=np.int64).reshape(-1)))
        n = rows_arr.size
        Z = np.zeros((n, N), dtype=np.float64)
        A = np.zeros((n, K), dtype=np.float64) if return_softmax else None
        rc = fn(X.ctypes.data, Y.ctypes.data, M, K, N, rows_arr.ctypes.data if n else None, n,
                Z.ctypes.data, A.ctypes.data if A is not None else None, int(threads))
        if rc == 4:
            raise OracleDomainError(ERRORS[4])
        if rc != 0:
            raise RuntimeError("oracle returned error code %d (%s)" % (rc, ERRORS.get(rc, "?")))
        return (Z, A) if return_softmax else Z


_DEFAULT: Optional[SoftmaxMatmulOracle] = None


def default_oracle() -> SoftmaxMatmulOracle:
    """The oracle built from ``softmax_matmul_oracle.c`` (compiled on first use
    if absent or older than its source)."""
    global _DEFAULT
    if _DEFAULT is None:
        if (not os.path.exists(LIBRARY)
                or os.path.getmtime(LIBRARY) < os.path.getmtime(SOURCE)):
            build()
        _DEFAULT = SoftmaxMatmulOracle(LIBRARY)
    return _DEFAULT


def softmax_matmul_rows(X, Y, rows=None, threads: int = 0, return_softmax: bool = False):
    return default_oracle().rows(X, Y, rows=rows, threads=threads, return_softmax=return_softmax)
