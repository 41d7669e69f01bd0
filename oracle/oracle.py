"""ctypes wrapper around the C fp64 oracle (``gmlp_oracle.c``).

TEST INFRASTRUCTURE ONLY: nothing on the product path may import this module.

The oracle evaluates the plain definition of the SiLU Gated MLP
(Fig. fig:mlp-example, Section 4.2; matmul semantics Fig. fig:op-sema,
Section 4.2.1; silu(x) = x * sigmoid(x), table tab:nki-ops, Section 5.1)
in IEEE double precision, on a chosen subset of rows of X, and its variants:
the gate activation swish_beta(g) = g * sigmoid(beta g) (SwiGLU) or
sigmoid(g) (GLU), and RMSNorm in front (Section 2: each row x becomes
x / sqrt(mean(x^2) + eps)).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "gmlp_oracle.c")
LIBRARY = os.path.join(HERE, "liboracle.so")

# Plain IEEE double arithmetic: no contraction into fused multiply-add, no
# fast-math.  x86-64-v3 (AVX2) lets gcc vectorise across output columns, which
# does not change any element's accumulation order.
CFLAGS = ["-O3", "-march=x86-64-v3", "-ffp-contract=off", "-fopenmp", "-fPIC",
          "-shared", "-Wall", "-Wextra"]


def build(source: str = SOURCE, output: str = LIBRARY, extra_flags: Sequence[str] = ()) -> str:
    """Compile ``source`` into the shared library ``output`` with gcc."""
    tmp = output + ".tmp%d" % os.getpid()
    cmd = ["gcc", *CFLAGS, *extra_flags, "-o", tmp, source, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, output)
    return output


_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_D = ctypes.c_double
_INT = ctypes.c_int

# Gate activations (the values of the library's enum gmlp_activation).
ACTIVATIONS = {"silu": 0, "swish": 1, "sigmoid": 2}


class Oracle:
    """One loaded copy of the oracle library."""

    def __init__(self, path: str = LIBRARY):
        self.path = path
        lib = ctypes.CDLL(path)
        lib.gmlp_oracle_silu.argtypes = [ctypes.c_double]
        lib.gmlp_oracle_silu.restype = ctypes.c_double
        lib.gmlp_oracle_bf16_to_f64.argtypes = [ctypes.c_uint16]
        lib.gmlp_oracle_bf16_to_f64.restype = ctypes.c_double
        lib.gmlp_oracle_sigmoid.argtypes = [_D]
        lib.gmlp_oracle_sigmoid.restype = _D
        lib.gmlp_oracle_gate.argtypes = [_D, _INT, _D]
        lib.gmlp_oracle_gate.restype = _D
        for name in ("gmlp_oracle_rows_bf16", "gmlp_oracle_rows_f64"):
            fn = getattr(lib, name)
            fn.argtypes = [_P, _P, _P, _P, _I64, _I64, _I64, _P, _I64, _P, _P, _INT]
            fn.restype = _INT
        for name in ("gmlp_oracle_variant_rows_bf16", "gmlp_oracle_variant_rows_f64"):
            fn = getattr(lib, name)
            fn.argtypes = [_P, _P, _P, _P, _I64, _I64, _I64, _INT, _D, _INT, _D, _P, _I64, _P, _P,
                           _INT]
            fn.restype = _INT
        lib.gmlp_oracle_down_rows_bf16.argtypes = [_P, _P, _I64, _I64, _I64, _P, _I64, _P,
                                                   ctypes.c_int]
        lib.gmlp_oracle_down_rows_bf16.restype = ctypes.c_int
        lib.gmlp_oracle_max_threads.argtypes = []
        lib.gmlp_oracle_max_threads.restype = ctypes.c_int
        self.lib = lib

    # -- scalar helpers ---------------------------------------------------
    def silu(self, z):
        """silu(z) = z * sigmoid(z), elementwise, in double precision."""
        arr = np.asarray(z, dtype=np.float64)
        out = np.vectorize(self.lib.gmlp_oracle_silu, otypes=[np.float64])(arr)
        return float(out) if np.ndim(z) == 0 else out

    def sigmoid(self, z):
        arr = np.asarray(z, dtype=np.float64)
        out = np.vectorize(self.lib.gmlp_oracle_sigmoid, otypes=[np.float64])(arr)
        return float(out) if np.ndim(z) == 0 else out

    def gate(self, g, activation: str = "silu", beta: float = 1.0):
        """act(g) of the named gate activation, elementwise."""
        act = ACTIVATIONS[activation]
        arr = np.asarray(g, dtype=np.float64)
        out = np.vectorize(lambda v: self.lib.gmlp_oracle_gate(v, act, beta), otypes=[np.float64])(arr)
        return float(out) if np.ndim(g) == 0 else out

    def bf16_to_f64(self, bits):
        arr = np.asarray(bits, dtype=np.uint16)
        return np.vectorize(self.lib.gmlp_oracle_bf16_to_f64, otypes=[np.float64])(arr)

    def max_threads(self) -> int:
        return int(self.lib.gmlp_oracle_max_threads())

    # -- the Gated MLP ----------------------------------------------------
    def gated_mlp_rows(self, X, Wg, Wu, Wd, rows: Optional[Sequence[int]] = None,
                       threads: int = 0, return_h: bool = False, activation: str = "silu",
                       beta: float = 1.0, rmsnorm: bool = False, eps: float = 1e-6):
        """Rows of Y = (act(X Wg) * (X Wu)) Wd in double precision.

        X [T, D], Wg [D, F], Wu [D, F], Wd [F, D]: either all ``uint16``
        (bf16 bit patterns, decoded exactly) or all floating point (converted
        to float64).  ``rows`` selects rows of X (default: all).  act is
        silu (default), swish (g * sigmoid(beta g)) or sigmoid; ``rmsnorm``
        replaces each row x of X by x / sqrt(mean(x^2) + eps) first.  Returns
        Y [len(rows), D] (and H [len(rows), F] if ``return_h``).
        """
        arrays = [np.asarray(a) for a in (X, Wg, Wu, Wd)]
        plain = activation == "silu" and not rmsnorm
        if all(a.dtype == np.uint16 for a in arrays):
            fn = self.lib.gmlp_oracle_rows_bf16 if plain else self.lib.gmlp_oracle_variant_rows_bf16
            arrays = [np.ascontiguousarray(a, dtype=np.uint16) for a in arrays]
        elif not any(a.dtype == np.uint16 for a in arrays):
            fn = self.lib.gmlp_oracle_rows_f64 if plain else self.lib.gmlp_oracle_variant_rows_f64
            arrays = [np.ascontiguousarray(a, dtype=np.float64) for a in arrays]
        else:
            raise TypeError("mixing bf16 bit patterns and floating-point inputs")
        X, Wg, Wu, Wd = arrays
        if X.ndim != 2 or Wg.ndim != 2 or Wu.ndim != 2 or Wd.ndim != 2:
            raise ValueError("all operands must be 2-D")
        T, D = X.shape
        F = Wg.shape[1]
        if Wg.shape != (D, F) or Wu.shape != (D, F) or Wd.shape != (F, D):
            raise ValueError("shape mismatch: X %s Wg %s Wu %s Wd %s"
                             % (X.shape, Wg.shape, Wu.shape, Wd.shape))
        if rows is None:
            rows_arr = np.arange(T, dtype=np.int64)
        else:
            rows_arr = np.ascontiguousarray(np.asarray(rows, dtype=np.int64).reshape(-1))
        n = rows_arr.size
        Y = np.zeros((n, D), dtype=np.float64)
        H = np.zeros((n, F), dtype=np.float64) if return_h else None
        tail = (rows_arr.ctypes.data if n else None, n, Y.ctypes.data,
                H.ctypes.data if H is not None else None, int(threads))
        if plain:
            rc = fn(X.ctypes.data, Wg.ctypes.data, Wu.ctypes.data, Wd.ctypes.data, T, D, F, *tail)
        else:
            rc = fn(X.ctypes.data, Wg.ctypes.data, Wu.ctypes.data, Wd.ctypes.data, T, D, F,
                    ACTIVATIONS[activation], float(beta), int(bool(rmsnorm)), float(eps), *tail)
        if rc != 0:
            raise RuntimeError("oracle returned error code %d" % rc)
        return (Y, H) if return_h else Y


    def down_rows(self, H, Wd, rows: Optional[Sequence[int]] = None, threads: int = 0):
        """Rows of H Wd in double precision for bf16 bit patterns H [T, F] and
        Wd [F, D] (the down projection alone)."""
        H = np.ascontiguousarray(H, dtype=np.uint16)
        Wd = np.ascontiguousarray(Wd, dtype=np.uint16)
        T, F = H.shape
        if Wd.shape[0] != F:
            raise ValueError("shape mismatch: H %s Wd %s" % (H.shape, Wd.shape))
        D = Wd.shape[1]
        rows_arr = (np.arange(T, dtype=np.int64) if rows is None
                    else np.ascontiguousarray(np.asarray(rows, dtype=np.int64).reshape(-1)))
        n = rows_arr.size
        Y = np.zeros((n, D), dtype=np.float64)
        rc = self.lib.gmlp_oracle_down_rows_bf16(H.ctypes.data, Wd.ctypes.data, T, F, D,
                                                 rows_arr.ctypes.data if n else None, n,
                                                 Y.ctypes.data, int(threads))
        if rc != 0:
            raise RuntimeError("oracle returned error code %d" % rc)
        return Y


_DEFAULT: Optional[Oracle] = None


def default_oracle() -> Oracle:
    """The oracle built from ``gmlp_oracle.c`` (compiled on first use if absent
    or older than its source)."""
    global _DEFAULT
    if _DEFAULT is None:
        if (not os.path.exists(LIBRARY)
                or os.path.getmtime(LIBRARY) < os.path.getmtime(SOURCE)):
            build()
        _DEFAULT = Oracle(LIBRARY)
    return _DEFAULT


def silu(z):
    return default_oracle().silu(z)


def gated_mlp_rows(X, Wg, Wu, Wd, rows=None, threads: int = 0, return_h: bool = False,
                   **variant):
    return default_oracle().gated_mlp_rows(X, Wg, Wu, Wd, rows=rows, threads=threads,
                                           return_h=return_h, **variant)
